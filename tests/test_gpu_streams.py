"""Calls on different streams at the same time, each with its own workspace.

A handle holds host memory only and the kernels keep their counters and partial
results in the workspace, so calls on different streams may overlap as long as
their workspaces differ.  Here a decode call and a multi-token call from one handle
run on two streams (default priority), ten times each without waiting in between,
and every result is compared with the fp64 oracle afterwards.
"""
import numpy as np
import pytest

import oracle
from paper_2607_09207_amd import inputs as I
from test_gpu_parity import assert_close, handle_for, log, torch_cuda  # noqa: F401  (the fixture)

pytestmark = pytest.mark.gpu


def test_two_streams_with_their_own_workspaces(torch_cuda):
    torch = torch_cuda
    wa = I.make_custom([3000, 20, 1700, 9, 800, 5000, 1], 28, 4, 128, seed=61)
    wb = I.make_multi([900, 64, 2200, 17], [300, 64, 128, 17], 28, 4, 128, seed=62,
                      max_pages_per_seq=wa.max_pages_per_seq)
    h = handle_for(wa, max_batch=8)
    ta, tb = I.to_torch(wa, "cuda"), I.to_torch(wb, "cuda")
    qs = torch.from_numpy(np.ascontiguousarray(wb.q_start, np.int32)).cuda()
    wsa = torch.zeros(h.workspace_bytes + 256, dtype=torch.uint8, device="cuda")
    wsb = torch.zeros(h.workspace_bytes + 256, dtype=torch.uint8, device="cuda")
    oa = torch.empty((wa.batch, wa.num_q_heads, wa.head_dim), dtype=torch.float32, device="cuda")
    ob = torch.empty((int(wb.q_start[-1]), wb.num_q_heads, wb.head_dim), dtype=torch.float32, device="cuda")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    log("two streams: decode B=7 on one, multi-token B=4 on the other, 10 rounds")
    for _ in range(10):
        h(ta["q"], ta["k_cache"], ta["v_cache"], ta["block_table"], ta["seq_lens"], out=oa, workspace=wsa, stream=sa)
        h.multi(tb["q"], tb["k_cache"], tb["v_cache"], tb["block_table"], tb["seq_lens"], qs, out=ob, workspace=wsb,
                stream=sb)
    torch.cuda.synchronize()
    assert h.read_flags(workspace=wsa, device=oa.device) == 0
    assert h.read_flags(workspace=wsb, device=ob.device) == 0
    assert_close(oa.double().cpu().numpy(), oracle.run(wa), "bf16", "decode on stream a")
    assert_close(ob.double().cpu().numpy(), oracle.run_multi(wb), "bf16", "multi-token on stream b")
