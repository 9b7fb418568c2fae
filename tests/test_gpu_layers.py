"""GPU parity of the multi-layer transitions (ekv_demote_layers /
ekv_refine_layers): the same pairs in every layer's pool in one launch.
Per layer the oracle's single-layer demote / refine defines the result
(the layers share the block table); every pool byte, the refinement bytes
of every layer, the block table, tags and freed ids: bit-exact."""

import numpy as np
import pytest

from oracle import transitions as otr
from paper_2609_33536_amd import ekv, workloads
from tests.gpu_util import host_safety_check, require_gpu

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("num_layers,hkv", [(1, 2), (3, 2), (5, 8)])
def test_demote_refine_all_layers(num_layers, hkv):
    torch = require_gpu()
    lens = [300, 1024, 77, 640, 2000]
    case = workloads.make_decode_case(lens, 4 * hkv, hkv, seed=50 + num_layers, base_fraction=0.5,
                                      spare_blocks=40)
    host_safety_check(case, case["pool"].shape)
    rng = np.random.default_rng(60 + num_layers)
    pools = [case["pool"]] + [workloads.to_words(rng.standard_normal(case["pool"].shape, dtype=np.float32), "bf16")
                              for _ in range(num_layers - 1)]
    dev = [torch.from_numpy(p.view(np.int16).copy()).cuda() for p in pools]
    layer_kv = torch.tensor([t.data_ptr() for t in dev], dtype=torch.int64, device="cuda")
    pool = ekv.make_pool(dev[0], hkv, "bf16")
    pairs = case["pairs"]
    n = len(pairs)
    assert n > 0
    bt = torch.from_numpy(case["block_table"].copy()).cuda()
    tags = torch.from_numpy(case["tags"].copy()).cuda()
    pairs_d = torch.from_numpy(pairs.copy()).cuda()
    block_bytes = 2 * hkv * 16 * 128 * 2
    freed = torch.empty(n, dtype=torch.int32, device="cuda")
    lo = torch.empty((n, num_layers, block_bytes), dtype=torch.uint8, device="cuda")
    print(f"demote_layers: L={num_layers} Hkv={hkv} pairs={n}", flush=True)
    ekv.demote_layers(pool, layer_kv, pairs_d, bt, tags, freed, lo)
    torch.cuda.synchronize()
    opools, olos = [], []
    for p in pools:
        op, obt, otg, ofreed, olo = otr.demote(p, case["block_table"], case["tags"], pairs, case["seq_lens"])
        opools.append(op)
        olos.append(olo)
    assert np.array_equal(bt.cpu().numpy(), obt)
    assert np.array_equal(tags.cpu().numpy(), otg)
    assert np.array_equal(freed.cpu().numpy(), ofreed)
    lo_h = lo.cpu().numpy()
    for layer in range(num_layers):
        assert np.array_equal(dev[layer].cpu().numpy().view(np.uint16), opools[layer]), layer
        assert np.array_equal(lo_h[:, layer].reshape(olos[layer].shape), olos[layer]), layer

    # refinement of every layer from its own refinement bytes
    fifo = otr.FreeFifo(case["free"])
    fifo.commit_freed(ofreed)
    new = fifo.acquire(n)
    new_d = torch.from_numpy(new).cuda()
    print(f"refine_layers: L={num_layers} Hkv={hkv} pairs={n}", flush=True)
    ekv.refine_layers(pool, layer_kv, pairs_d, new_d, bt, tags, lo)
    torch.cuda.synchronize()
    for layer in range(num_layers):
        rp, rbt, rtg = otr.refine(opools[layer], obt, otg, pairs, new, olos[layer], case["seq_lens"])
        assert np.array_equal(dev[layer].cpu().numpy().view(np.uint16), rp), layer
    assert np.array_equal(bt.cpu().numpy(), rbt)
    assert np.array_equal(tags.cpu().numpy(), rtg)


def test_layers_argument_errors():
    torch = require_gpu()
    case = workloads.make_decode_case([64, 64], 8, 2, seed=8, base_fraction=1.0, spare_blocks=2)
    dev = torch.from_numpy(case["pool"].view(np.int16).copy()).cuda()
    pool = ekv.make_pool(dev, 2, "bf16")
    bt = torch.from_numpy(case["block_table"].copy()).cuda()
    tags = torch.from_numpy(case["tags"].copy()).cuda()
    pairs = torch.from_numpy(case["pairs"].copy()).cuda()
    freed = torch.empty(len(case["pairs"]), dtype=torch.int32, device="cuda")
    empty = torch.empty(0, dtype=torch.int64, device="cuda")
    with pytest.raises(ekv.EkvError):
        ekv.demote_layers(pool, empty, pairs, bt, tags, freed)       # no layers
    torch.cuda.synchronize()
    assert np.array_equal(dev.cpu().numpy().view(np.uint16), case["pool"])   # nothing was enqueued
