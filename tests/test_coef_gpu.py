"""GPU parity of the App. D.1 per-chunk coefficient records: the record the
library writes is byte-equal to the oracle's, for chunks from all rows kept
(dense) to none kept (sparse, counts only), and unpacking it into a cache
whose chunk rows hold garbage restores them and changes nothing else."""
import numpy as np
import pytest
import torch

import oracle
import packed
import synth

pytestmark = pytest.mark.gpu

from paper_2609_26425_amd import quantwm as qw  # noqa: E402  (fails loudly if the library is missing)

DEV = "cuda:0"

# two batches, three heads, r = 12 (rows of 12 bytes), 1000 slots
WL = synth.Workload(name="coef-ragged", dtype="bf16", batch=2, heads=3, head_dim=128, n_cache=1000, n_q=300,
                    q_start=700, frame_tokens=50, n_centroids=37, group_size=32, rank=12, top_m=3, q_rank=8,
                    n_out=4, out_scale=10.0, n_hist=500, chunk=300, seed=7)

_state = {}


def _say(msg):
    print(msg, flush=True)


def _encoded():
    if not _state:
        cfg = oracle.cfg_from_workload(WL)
        k = synth.round_to(synth.tensor(WL, "k", WL.n_cache), "bf16")
        v = synth.round_to(synth.tensor(WL, "v", WL.n_cache), "bf16")
        qh = synth.round_to(synth.tensor(WL, "qhist", WL.n_hist), "bf16")
        tables = oracle.calibrate(cfg, qh, np.ascontiguousarray(k[:, :WL.chunk]),
                                  np.ascontiguousarray(v[:, :WL.chunk]), WL.kmeans_iters)
        cache = oracle.new_cache(cfg)
        oracle.append(cfg, tables, cache, 0, k, v)
        _state.update(cfg=cfg, cache=cache)
    return _state["cfg"], _state["cache"]


def _gpu_cfg():
    return qw.make_config(WL.batch, WL.heads, WL.head_dim, WL.n_centroids, WL.group_size, WL.rank, WL.top_m,
                          WL.capacity, "bf16")


@pytest.mark.parametrize("keep", [0.0, 0.05, 0.4, 0.75, 1.0])
@pytest.mark.parametrize("start,n", [(0, 1000), (300, 700), (37, 1), (512, 0)])
def test_coef_record_parity(keep, start, n):
    ocfg, base = _encoded()
    nbh = WL.batch * WL.heads
    lay = packed.layout(WL.batch, WL.heads, WL.head_dim, WL.group_size, WL.rank, WL.capacity)
    cache = base.copy()
    r = np.random.default_rng(int(keep * 100) + start)
    for bh in range(nbh):
        packed.zero_coef_rows(cache, lay, bh, np.nonzero(r.random(WL.n_cache) >= keep)[0])
    want = oracle.coef_pack(ocfg, cache, start, n)
    _say(f"[case] keep {keep} chunk [{start}, {start + n}): oracle record {want.size} B")
    cfg = _gpu_cfg()
    cache_d = torch.from_numpy(cache).to(DEV)
    rec = torch.zeros(qw.quantwm_coef_record_max_bytes(cfg, n), dtype=torch.uint8, device=DEV)
    written, layout = qw.quantwm_coef_pack(cfg, cache_d, start, n, rec)
    torch.cuda.synchronize()
    assert written == want.size and layout == int(want[:4].view("<u4")[0])
    got = rec.cpu().numpy()
    assert np.array_equal(got[:written], want), "record bytes differ from the oracle's"
    assert np.array_equal(cache_d.cpu().numpy(), cache), "packing changed the cache"
    target = np.random.default_rng(3).integers(0, 256, cache.size, dtype=np.uint8)
    target_d = torch.from_numpy(target).to(DEV)
    qw.quantwm_coef_unpack(cfg, rec, target_d, start, n, record_bytes=written)
    torch.cuda.synchronize()
    back = target_d.cpu().numpy()
    chunk = packed.coef_byte_mask(lay, nbh, start, n)
    assert np.array_equal(back[chunk], cache[chunk]) and np.array_equal(back[~chunk], target[~chunk])
    _say(f"[ok] keep {keep} chunk [{start}, {start + n}): {'sparse' if layout else 'dense'} {written} B")


def test_coef_unpack_rejects_a_mismatched_or_truncated_record():
    ocfg, cache = _encoded()
    cfg = _gpu_cfg()
    rec = torch.from_numpy(oracle.coef_pack(ocfg, cache, 100, 200)).to(DEV)
    target = torch.zeros(cache.size, dtype=torch.uint8, device=DEV)
    for start, n, nbytes, msg in [(100, 199, rec.numel(), "does not match"), (100, 200, rec.numel() - 1, "truncated")]:
        with pytest.raises(qw.QuantwmError) as e:
            qw.quantwm_coef_unpack(cfg, rec, target, start, n, record_bytes=nbytes)
        assert e.value.status == qw.ERR_INVALID_ARG and msg in qw.quantwm_last_error()
    torch.cuda.synchronize()
    assert not target.any()


@pytest.mark.timeout(600)
def test_coef_record_full_size():
    # The LingBot-shaped append chunk (40 heads, 4,680 tokens at slot 28,080,
    # r = 16), encoded by the oracle, with 30% of the rows dropped as the gate
    # leaves them: the library's record equals the oracle's, and unpacking it
    # restores the chunk.
    wl = synth.WORKLOADS["lingbot-40h"]
    start, n = wl.n_cache - wl.chunk, wl.chunk
    ocfg = oracle.cfg_from_workload(wl)
    k = synth.round_to(synth.tensor(wl, "k", n, start=start), "bf16")
    v = synth.round_to(synth.tensor(wl, "v", n, start=start), "bf16")
    qh = synth.round_to(synth.tensor(wl, "qhist", 256), "bf16")  # the record does not depend on table quality
    tables = oracle.calibrate(ocfg, qh, k, v, 1)
    cache = oracle.new_cache(ocfg)
    oracle.append(ocfg, tables, cache, start, k, v)
    nbh = wl.batch * wl.heads
    lay = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity)
    r = np.random.default_rng(11)
    for bh in range(nbh):
        packed.zero_coef_rows(cache, lay, bh, start + np.nonzero(r.random(n) < 0.3)[0])
    want = oracle.coef_pack(ocfg, cache, start, n)
    _say(f"[case] lingbot-40h chunk [{start}, {start + n}): oracle record {want.size} B")
    cfg = qw.make_config(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m,
                         wl.capacity, "bf16")
    cache_d = torch.from_numpy(cache).to(DEV)
    rec = torch.zeros(qw.quantwm_coef_record_max_bytes(cfg, n), dtype=torch.uint8, device=DEV)
    written, layout = qw.quantwm_coef_pack(cfg, cache_d, start, n, rec)
    torch.cuda.synchronize()
    assert written == want.size and np.array_equal(rec.cpu().numpy()[:written], want)
    target = torch.zeros_like(cache_d)
    qw.quantwm_coef_unpack(cfg, rec, target, start, n, record_bytes=written)
    torch.cuda.synchronize()
    chunk = packed.coef_byte_mask(lay, nbh, start, n)
    back = target.cpu().numpy()
    assert np.array_equal(back[chunk], cache[chunk]) and not back[~chunk].any()
    _say(f"[ok] lingbot-40h chunk: {'sparse' if layout else 'dense'} {written} B of "
         f"{qw.quantwm_coef_record_max_bytes(cfg, n)} B")
