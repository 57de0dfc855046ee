"""The decode call captured in a HIP graph (torch.cuda.graph) and replayed.

Neither entry point allocates, clears memory or synchronises inside a call, and
both leave their counters at zero when the kernel ends, so a captured call replays
as often as the caller likes: here the workspace entry point (workspace zeroed once,
before capture) and the no-allocation entry point are captured together and the
graph is replayed four times, with eager work and synchronisation between the
replays; every replay must equal the eager call bit for bit.
"""
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
