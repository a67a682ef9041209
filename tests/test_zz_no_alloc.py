"""The no-allocation ids partition (ids_partition_static) against the
workspace-taking ids_partition, through the C ABI.

Integer work, so bit-exact: keys, shard offsets, inverse and info.  Two calls
in a row on the same GPU -- the full one-million-id benchmark input, then a
smaller ragged batch -- so the second call runs over the array the first one
left behind.  The size limit is checked on the host.
"""
import numpy as np
import pytest
import torch

from paper_2509_20883_amd import recis as R
from paper_2509_20883_amd import workloads as W


def _log(*a):
    print(*a, flush=True)


def _outputs(n, G, dev):
    return (torch.empty(max(n, 1), dtype=torch.int64, device=dev), torch.empty(G + 1, dtype=torch.int64, device=dev),
            torch.empty(max(n, 1), dtype=torch.int32, device=dev), torch.empty(2, dtype=torch.int64, device=dev))


def _static(v, G, seed):
    n = v.numel()
    keys, offs, inv, info = _outputs(n, G, v.device)
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    R.ids_partition_static(v, G, seed, keys, offs, inv, info)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before  # the call took nothing from torch's allocator
    U = int(info[0].item())
    return keys[:U].cpu().numpy(), offs.cpu().numpy(), inv[:n].cpu().numpy(), info.cpu().numpy()


def _reference(v, G, seed):
    keys, offs, inv, info = R.ids_partition(v, G, seed)
    torch.cuda.synchronize()
    U = int(info[0].item())
    return keys[:U].cpu().numpy(), offs.cpu().numpy(), inv.cpu().numpy(), info.cpu().numpy()


@pytest.mark.gpu
def test_static_matches_workspace_call_twice():
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    big = W.ids_partition_values(step=0)                     # the one-million-id benchmark input
    g = np.random.default_rng(7)
    small = (g.zipf(1.1, size=300003) % 50000).astype(np.int64) * 0x9E3779B1  # smaller, ragged tail
    for values, G, seed in ((big, 8, W.IDS_PARTITION_SEED), (small, 1000, 12345)):
        assert values.size <= R.IDS_STATIC_MAX_IDS
        _log(f"ids_partition_static n={values.size} G={G}")
        v = torch.from_numpy(values).to(dev)
        got = _static(v, G, seed)
        want = _reference(v, G, seed)
        for name, a, b in zip(("keys", "shard offsets", "inverse", "info"), got, want):
            assert np.array_equal(a, b), name
        assert int(got[3][1]) == 0 and got[1][-1] == got[3][0]


@pytest.mark.gpu
def test_static_empty_and_limit():
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    v = torch.empty(0, dtype=torch.int64, device=dev)
    keys, offs, inv, info = _outputs(0, 4, dev)
    R.ids_partition_static(v, 4, 1, keys, offs, inv, info)
    torch.cuda.synchronize()
    assert offs.cpu().tolist() == [0] * 5 and info.cpu().tolist() == [0, 0]
    # one id past the limit is refused on the host, before any GPU work
    lim = R.IDS_STATIC_MAX_IDS + 1
    v = torch.zeros(lim, dtype=torch.int64, device=dev)
    keys, offs, inv, info = _outputs(lim, 4, dev)
    with pytest.raises(R.RecisError) as e:
        R.ids_partition_static(v, 4, 1, keys, offs, inv, info)
    assert e.value.status == R.EINVAL
