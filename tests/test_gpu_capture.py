"""The layer enqueues without synchronising the host or allocating (paper
Section 3.1.1: routing metadata is built on the GPU with no stream
synchronisation): capturing moe_fused_fp8 into a HIP graph succeeds -- a
synchronisation or allocation inside the capture would fail it -- and each
replay, with other calls of the layer run eagerly in between, gives the eager
result bit for bit.  The graph is never timed."""
import pytest
import torch

import workloads as W
from gpu_helpers import inputs, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def M():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_14560_amd as M
    M.lib()
    return M


@pytest.mark.parametrize("name", ["decode", "mid", "small_t128", "prefill"])
def test_graph_capture_replays_eager_result(M, name):
    cfg = W.all_configs()[name]
    log(f"capture {name}")
    inp = inputs(cfg, 0)
    other = W.generate(cfg.with_(T=cfg.T), 1, device="cuda")
    s = M.Shape.of(cfg)
    ws = M.alloc_workspace(s)
    ro = M.alloc_route_out(s)
    out = torch.empty(cfg.T, cfg.H, dtype=torch.bfloat16, device="cuda")
    args = (inp.hidden, inp.hidden_scale, inp.logits, inp.bias, inp.w13, inp.w13_scale, inp.w2,
            inp.w2_scale)
    M.fused_fp8(s, *args, out=out, route_out=ro, workspace=ws)   # eager reference
    torch.cuda.synchronize()
    ref_out = out.clone()
    ref_ro = {k: v.clone() for k, v in ro.items()}

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=side):
        M.fused_fp8(s, *args, out=out, route_out=ro, workspace=ws)
    torch.cuda.synchronize()

    ws2 = M.alloc_workspace(s)
    out2 = torch.empty_like(out)
    for i in range(3):
        out.fill_(0)
        ro["topk_ids"].fill_(-7)
        # eager work on other inputs between replays
        M.fused_fp8(s, other.hidden, other.hidden_scale, other.logits, other.bias, inp.w13,
                    inp.w13_scale, inp.w2, inp.w2_scale, out=out2, workspace=ws2)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref_out.view(torch.int16)), f"replay {i}: out differs"
        P = int(ref_ro["expert_offsets"][-1])
        for k in ref_ro:
            n = P if k == "perm_token" else None
            assert torch.equal(ro[k][:n], ref_ro[k][:n]), f"replay {i}: {k} differs"
    log(f"capture {name}: 3 replays bit-identical")
