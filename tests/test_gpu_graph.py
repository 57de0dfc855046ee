"""The decode call captured in a HIP graph (torch.cuda.graph) and replayed.

Neither entry point allocates, clears memory or synchronises inside a call, and
both leave their counters at zero when the kernel ends, so a captured call replays
as often as the caller likes: here the workspace entry point (workspace zeroed once,
before capture) and the no-allocation entry point are captured together and the
graph is replayed four times, with eager work and synchronisation between the
replays; every replay must equal the eager call bit for bit.  The multi-token call
and both forms of the shared-prompt call (packed, one launch; prompt pass, two) are
captured and replayed the same way.
"""
import numpy as np
import pytest

import oracle
from paper_2607_09207_amd import inputs as I
from test_gpu_parity import assert_close, handle_for, log, torch_cuda  # noqa: F401  (the fixture)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kv,Hq,Hkv", [("bf16", 28, 4), ("fp8_e4m3fn", 64, 8)])
def test_captured_decode_calls_replay_like_the_eager_call(torch_cuda, kv, Hq, Hkv):
    torch = torch_cuda
    w = I.make_custom([3000, 20, 1700, 9, 800, 5000, 1], Hq, Hkv, 128, kv_dtype=kv, seed=71)
    h = handle_for(w)
    t = I.to_torch(w, "cuda")
    args = (t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"])
    kw = dict(k_scale=t["k_scale"], v_scale=t["v_scale"])
    ref = h(*args, **kw)                                  # eager, and warms up both entry points
    h.run_noalloc(*args, **kw)
    out = torch.empty_like(ref)
    out_na = torch.empty_like(ref)
    ws = torch.zeros(h.workspace_bytes + 256, dtype=torch.uint8, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        h(*args, **kw, out=out, workspace=ws)
        h.run_noalloc(*args, **kw, out=out_na, flags=flags)
    torch.cuda.synchronize()
    for r in range(4):
        out.zero_()
        out_na.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        log(f"graph replay {r} ({kv})")
        assert torch.equal(out, ref), f"replay {r}: workspace call differs from the eager call"
        assert torch.equal(out_na, ref), f"replay {r}: no-allocation call differs from the eager call"
    assert int(flags.item()) == 0
    assert h.read_flags(workspace=ws, device=out.device) == 0
    assert_close(out.double().cpu().numpy(), oracle.run(w), kv, f"graph replay ({kv})")


def test_captured_multi_token_and_grouped_calls_replay_like_the_eager_calls(torch_cuda):
    torch = torch_cuda
    wm = I.make_multi([900, 64, 2200, 17], [300, 64, 128, 17], 28, 4, 128, seed=72)
    lens = [256 + t for t in (0, 9, 400, 33, 70, 1, 16, 5)]
    wg = I.make_custom(lens, 12, 2, 128, seed=73, shared_prefix=(4, 256))
    hm, hg = handle_for(wm), handle_for(wg)
    tm, tg = I.to_torch(wm, "cuda"), I.to_torch(wg, "cuda")
    qs = torch.from_numpy(np.ascontiguousarray(wm.q_start, np.int32)).cuda()
    pp = torch.full((2,), 16, dtype=torch.int32, device="cuda")
    margs = (tm["q"], tm["k_cache"], tm["v_cache"], tm["block_table"], tm["seq_lens"], qs)
    gargs = (tg["q"], tg["k_cache"], tg["v_cache"], tg["block_table"], tg["seq_lens"])
    ref_m = hm.multi(*margs)
    ref_p = hg(*gargs, group_size=4, prefix_pages=pp)                          # packed
    ref_q = hg(*gargs, group_size=4, prefix_pages=pp, prompt_pages_hint=1 << 20)   # prompt pass
    om, op, oq = torch.empty_like(ref_m), torch.empty_like(ref_p), torch.empty_like(ref_q)
    wsm = torch.zeros(hm.workspace_bytes + 256, dtype=torch.uint8, device="cuda")
    wsp = torch.zeros(hg.grouped_workspace_bytes + 256, dtype=torch.uint8, device="cuda")
    wsq = torch.zeros(hg.grouped_workspace_bytes + 256, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=torch.cuda.Stream()):
        hm.multi(*margs, out=om, workspace=wsm)
        hg(*gargs, group_size=4, prefix_pages=pp, out=op, workspace=wsp)
        hg(*gargs, group_size=4, prefix_pages=pp, prompt_pages_hint=1 << 20, out=oq, workspace=wsq)
    torch.cuda.synchronize()
    for r in range(4):
        for o in (om, op, oq):
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        log(f"graph replay {r} (multi-token, packed, prompt pass)")
        assert torch.equal(om, ref_m), f"replay {r}: multi-token call differs from the eager call"
        assert torch.equal(op, ref_p), f"replay {r}: packed grouped call differs from the eager call"
        assert torch.equal(oq, ref_q), f"replay {r}: prompt-pass grouped call differs from the eager call"
    for h, ws in ((hm, wsm), (hg, wsp), (hg, wsq)):
        assert h.read_flags(workspace=ws, device=om.device) == 0
    assert_close(om.double().cpu().numpy(), oracle.run_multi(wm), "bf16", "graph multi-token")
    assert_close(oq.double().cpu().numpy(), oracle.run(wg), "bf16", "graph prompt pass")
