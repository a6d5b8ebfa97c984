"""GPU: replay_fill_synthetic writes, on the device, exactly the bytes and
side fields of the seeded host generator (dqn_inputs.frames, stacked four
frames per record, and the hashed side arrays): bit-exact over whole small
replays, a padded record stride and a record count that is not a multiple
of anything, and on sampled records of a full 1,000,000-transition replay."""
import numpy as np
import pytest

import dqn_inputs as di
import paper_1508_04186_amd as dq
from gpu_util import host, say

pytestmark = pytest.mark.gpu


def _alloc(size, c, stride, dev):
    import torch
    flat = torch.full((size * stride,), 0xAB, dtype=torch.uint8, device=dev)
    a = torch.empty(size, dtype=torch.uint8, device=dev)
    r = torch.empty(size, dtype=torch.int8, device=dev)
    t = torch.empty(size, dtype=torch.uint8, device=dev)
    return flat, dq.Replay(flat, a, r, t, size, c=c, record_stride=stride)


@pytest.mark.parametrize("size,c,pad,n_actions,seed", [
    (1, 4, 0, 6, 3),          # one record: frames 0..3
    (257, 4, 0, 6, 31),       # crosses two 100-frame segments
    (1013, 4, 48, 18, 1003),  # padded stride: the padding stays untouched
    (333, 1, 0, 3, 5),        # single-frame records
])
def test_fill_matches_host_generator(dev, size, c, pad, n_actions, seed):
    import torch
    say(f"[fill] size={size} c={c} pad={pad} A={n_actions} seed={seed}")
    rec = c * 84 * 84
    flat, rp = _alloc(size, c, rec + pad, dev)
    dq.replay_fill_synthetic(rp, n_actions, seed)
    torch.cuda.synchronize()
    got = host(flat).reshape(size, rec + pad)
    fr = di.frames(seed, 0, size + c - 1)
    want = np.stack([fr[i:i + c].reshape(-1) for i in range(size)])
    assert np.array_equal(got[:, :rec], want)
    assert (got[:, rec:] == 0xAB).all()
    a, r, t = di.side_arrays_hashed(size, n_actions, seed)
    assert np.array_equal(host(rp.action), a)
    assert np.array_equal(host(rp.reward), r)
    assert np.array_equal(host(rp.terminal), t)
    assert a.max() < n_actions and set(np.unique(r)) <= {-1, 0, 1}


def test_fill_full_size_sampled(dev):
    """The 1,000,000-transition replay of the large-network runs (26.3 GiB):
    64 sampled transitions, the first and the last, against the generator."""
    import torch
    size, seed, A = 1_000_000, 1003, 18
    say(f"[fill] full size {size} seed={seed}")
    rec = torch.empty((size, 4, 84, 84), dtype=torch.uint8, device=dev)
    a = torch.empty(size, dtype=torch.uint8, device=dev)
    r = torch.empty(size, dtype=torch.int8, device=dev)
    t = torch.empty(size, dtype=torch.uint8, device=dev)
    rp = dq.Replay(rec, a, r, t, size)
    dq.replay_fill_synthetic(rp, A, seed)
    torch.cuda.synchronize()
    idx = np.random.default_rng(9).integers(0, size - 1, 64).astype(np.int64)
    idx[:2] = [0, size - 2]
    s, sn, ra, rr, rt = di.transitions_at(seed, idx, A, size)
    ii = torch.from_numpy(idx).to(dev)
    assert np.array_equal(host(rec[ii]), s)
    assert np.array_equal(host(rec[ii + 1]), sn)
    assert np.array_equal(host(a[ii]).astype(np.int32), ra)
    assert np.array_equal(host(r[ii]).astype(np.float32), rr)
    assert np.array_equal(host(t[ii]), rt)
    # the side arrays in full, and the terminal rate of the stream
    ha, hr_, ht = di.side_arrays_hashed(size, A, seed)
    assert np.array_equal(host(a), ha) and np.array_equal(host(r), hr_) and np.array_equal(host(t), ht)
    assert 0.009 < ht.mean() < 0.011
    del rec
    torch.cuda.empty_cache()
