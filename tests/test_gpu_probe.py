"""GPU checks of the read-ceiling probe library (include/hbm_probe.h): the balanced
gather's claim protocol leaves its counter at zero after every launch, whatever the
split between static shares and claimed chunks, so launches can follow each other on
one counter; the readers write nothing but their sentinel words."""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def test_balanced_gather_leaves_its_counter_zero(torch_cuda):
    torch = torch_cuda
    from paper_2607_09207_amd import probe
    lib = probe.load()
    dev = "cuda"
    tile = 4096
    npages = 512
    k = torch.ones(npages * tile, dtype=torch.uint8, device=dev)
    v = torch.ones(npages * tile, dtype=torch.uint8, device=dev)
    rng = np.random.default_rng(5)
    n = 3000
    offs = torch.from_numpy(rng.integers(0, npages, size=n).astype(np.int64) * tile).to(dev)
    counter = torch.zeros(16, dtype=torch.int32, device=dev)
    sink = torch.zeros(64 * 64, dtype=torch.int32, device=dev)
    st = torch.cuda.current_stream().cuda_stream
    blocks, threads = 16, 256   # 64 waves
    waves = blocks * threads // 64
    for depth in (2, 3, 4):
        for chunk in (depth, 8, 64):
            for nd in (0, chunk * 7, (n // chunk) * chunk):
                nstatic = n - nd
                if 0 < nstatic and nstatic // waves < depth:
                    continue
                print(f"[probe] balanced gather depth={depth} chunk={chunk} nstatic={nstatic}", flush=True)
                for _ in range(2):
                    rc = lib.hbm_probe_tile_gather_balanced(k.data_ptr(), v.data_ptr(), offs.data_ptr(), n, nstatic,
                                                            chunk, counter.data_ptr(), tile, sink.data_ptr(), blocks,
                                                            threads, depth, st)
                    assert rc == 0
                    torch.cuda.synchronize()
                    assert int(counter[0].item()) == 0
    # Every loaded word is 0x01010101, so the folded value never equals the sentinel.
    assert int(sink.abs().sum().item()) == 0
