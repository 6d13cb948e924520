"""moe_fused_fp8_noalloc (the entry point for callers that cannot allocate)
against moe_fused_fp8 on the same inputs, through the C-ABI: two calls in a
row, the second with a smaller batch (so it runs on the library's scratch as
the first call left it), then a larger plan and a single token; outputs and
routing results must be identical bit for bit (the same kernels, fixed
summation orders).  A shape whose workspace exceeds the scratch is refused."""
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


def _both(M, cfg, seed):
    inp = inputs(cfg, seed)
    s = M.Shape.of(cfg)
    ro_a, ro_b = M.alloc_route_out(s), M.alloc_route_out(s)
    ref = M.fused_fp8(s, inp.hidden, inp.hidden_scale, inp.logits, inp.bias, inp.w13,
                      inp.w13_scale, inp.w2, inp.w2_scale, route_out=ro_a)
    out = torch.full((cfg.T, cfg.H), float("nan"), dtype=torch.bfloat16, device="cuda")
    M.fused_fp8_noalloc(s, inp.hidden, inp.hidden_scale, inp.logits, inp.bias, inp.w13,
                        inp.w13_scale, inp.w2, inp.w2_scale, out, route_out=ro_b)
    torch.cuda.synchronize()
    P = int(ro_a["expert_offsets"][-1])
    log(f"no-alloc T={cfg.T} seed {seed}: P={P}")
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"T={cfg.T}: outputs differ"
    for k in ro_a:
        n = P if k == "perm_token" else None
        assert torch.equal(ro_a[k][:n], ro_b[k][:n]), f"T={cfg.T}: {k} differs"


def test_noalloc_matches_workspace_entry_point(M):
    dec = W.CONFIGS["decode"]
    _both(M, dec, 0)                 # T = 16
    _both(M, dec.with_(T=5), 1)      # smaller, on the scratch the first call left
    _both(M, dec.with_(T=96), 2)     # a larger plan (no gate/up split)
    _both(M, dec.with_(T=1), 3)


def test_noalloc_refuses_shapes_beyond_its_scratch(M):
    cfg = W.CONFIGS["mid"]           # T = 256 needs a 76 MiB workspace
    inp = inputs(cfg, 0)
    s = M.Shape.of(cfg)
    out = torch.zeros(cfg.T, cfg.H, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(M.MoEError) as e:
        M.fused_fp8_noalloc(s, inp.hidden, inp.hidden_scale, inp.logits, inp.bias, inp.w13,
                            inp.w13_scale, inp.w2, inp.w2_scale, out)
    assert e.value.code == M.MOE_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert (out == 0).all()          # nothing was enqueued
