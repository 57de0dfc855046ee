"""The Python binding rejects tensors that do not match the handle (device, dtype,
shape, layout) before anything is launched: the kernels index every array by the
handle's configuration, so a mismatch would otherwise read or write out of bounds."""
import numpy as np
import pytest

import oracle
from paper_2607_09207_amd import RldaError
from paper_2607_09207_amd import inputs as I
from test_gpu_parity import assert_close, handle_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_09207_amd import _abi
    _abi.load()
    return torch


def bad(fn, *a, **kw):
    with pytest.raises(RldaError) as e:
        fn(*a, **kw)
    assert e.value.status == -1
    return str(e.value)


def test_decode_call_checks(torch_cuda):
    torch = torch_cuda
    w = I.make_custom([40, 300, 20], 8, 2, 128, seed=16)
    t = I.to_torch(w, "cuda")
    h = handle_for(w)
    q, k, v, bt, sl = t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"]
    assert "q must be" in bad(h, q.float(), k, v, bt, sl)
    assert "contiguous" in bad(h, q.transpose(1, 2).contiguous().transpose(1, 2), k, v, bt, sl)
    assert "out must be" in bad(h, q, k, v, bt, sl, out=torch.empty((3, 8, 128), dtype=torch.bfloat16, device="cuda"))
    assert "out must have shape" in bad(h, q, k, v, bt, sl, out=torch.empty((2, 8, 128), device="cuda"))
    assert "block_table" in bad(h, q, k, v, bt[:, :-1].contiguous(), sl)
    assert "block_table" in bad(h, q, k, v, bt.long(), sl)
    assert "seq_lens" in bad(h, q, k, v, bt, sl[:2].contiguous())
    assert "k_cache" in bad(h, q, k[:, :1].contiguous(), v, bt, sl)
    assert "pages" in bad(h, q, k, v, bt, sl, num_pages=k.shape[0] + 1)
    assert "strides" in bad(h, q, k.transpose(1, 2).contiguous().transpose(1, 2), v, bt, sl)
    assert "GPU" in bad(h, q.cpu(), k, v, bt, sl)
    assert "workspace" in bad(h, q, k, v, bt, sl, workspace=torch.zeros(h.workspace_bytes + 256, device="cuda"))
    assert "prefix_pages" in bad(h, q, k, v, bt, sl, group_size=2,
                                 prefix_pages=torch.zeros(1, dtype=torch.int32, device="cuda"))
    assert "flags" in bad(h.run_noalloc, q, k, v, bt, sl, flags=torch.zeros(2, dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()


def test_fp8_scales_multi_and_append_checks(torch_cuda):
    torch = torch_cuda
    w = I.make_multi([40, 30], [4, 2], 8, 2, 128, kv_dtype="fp8_e4m3fn", seed=5)
    t = I.to_torch(w, "cuda")
    h = handle_for(w)
    q, k, v, bt, sl = t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"]
    qs = torch.from_numpy(np.asarray(w.q_start, np.int32)).cuda()
    assert "k_scale" in bad(h.multi, q, k, v, bt, sl, qs, v_scale=t["v_scale"])
    assert "v_scale" in bad(h.multi, q, k, v, bt, sl, qs, k_scale=t["k_scale"], v_scale=t["v_scale"][:, :1].contiguous())
    assert "q_start" in bad(h.multi, q, k, v, bt, sl, qs.long(), k_scale=t["k_scale"], v_scale=t["v_scale"])
    # the batch comes from q_start: a shorter one no longer matches the block table
    assert "block_table" in bad(h.multi, q, k, v, bt, sl, qs[:2].contiguous(), k_scale=t["k_scale"],
                                v_scale=t["v_scale"])
    kn = torch.zeros((2, 2, 128), dtype=torch.bfloat16, device="cuda")
    assert "k_new" in bad(h.append, kn[:, :1].contiguous(), kn, k, v, bt, sl, k_scale=t["k_scale"],
                          v_scale=t["v_scale"])
    assert "v_new" in bad(h.append, kn, kn.float(), k, v, bt, sl, k_scale=t["k_scale"], v_scale=t["v_scale"])
    torch.cuda.synchronize()


def test_single_kv_head_in_the_slot_major_layout_is_accepted(torch_cuda):
    """torch may report any stride for a dimension of size 1 (here the one KV head of a
    [page][slot][head][d] cache); the binding checks only the strides of longer
    dimensions, which are the ones the kernels step through."""
    w = I.to_page_slot_head(I.make_custom([40, 300, 20, 1], 8, 1, 128, seed=17))
    t = I.to_torch(w, "cuda")
    h = handle_for(w)
    out = h(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"])
    torch_cuda.cuda.synchronize()
    assert h.read_flags(device=out.device) == 0
    assert_close(out.double().cpu().numpy(), oracle.run(w), "bf16", "one KV head, slot-major layout")

