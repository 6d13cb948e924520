"""GEMM1 pinned to integer arithmetic through the real kernels (paper Section
3.1.1, stage (3)), with no model of any accumulator.

Inputs are chosen so that every step before the re-quantisation is exact in
fp32 whatever the summation order: hidden codes are integers 5..16 with block
scales 1 or 2; each gate row holds 8 weights of 1.0 (scale 0.5), so every gate
value g is a multiple of 0.5 in [20, 128]; each up row holds +-1 on half its
positions (scale 0.25 or 0.5), so |u| <= 8192 is a multiple of 0.25.  Every
product fits the FP8 matrix cores' block sum exactly, the promotion by
power-of-two scales is exact, sigmoid(g) rounds to exactly 1 in fp32 for
g >= 20, so SwiGLU is g * u exactly (|g u| <= 2^20, a multiple of 1/8).  The
device's FP8 intermediate must then equal, bit for bit, the re-quantisation of
an int64 matrix product -- on every GEMM1 kernel the plan can pick (the batch
sizes below give 2 .. 400 rows per expert) -- and the output must meet the
plain tolerance with no flips."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import inputs, layer_parity, log, oracle_route

pytestmark = pytest.mark.gpu

BASE = W.MoEConfig("exact", T=8, H=1024, I=512, num_experts=16, num_local_experts=16,
                   local_expert_offset=0, n_group=4, topk_group=2, top_k=4)


@pytest.fixture(scope="module")
def M():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_14560_amd as M
    M.lib()
    return M


def _code(v):
    return torch.tensor([float(v)]).to(torch.float8_e4m3fn).view(torch.uint8).item()


def exact_inputs(cfg, seed):
    """Integer-valued inputs (see the module docstring) on the GPU, plus the
    integer values the test recomputes the intermediate from."""
    rng = np.random.default_rng(seed)
    H, I, El = cfg.H, cfg.I, cfg.num_local_experts
    xv = rng.integers(5, 17, (cfg.T, H))
    sx = np.exp2(rng.integers(0, 2, (cfg.T, H // 128))).astype(np.float32)
    codes = np.zeros(33, np.uint8)
    for v in range(-16, 17):
        codes[v + 16] = _code(v)
    gate = np.zeros((El, I, H), np.int64)
    for e in range(El):
        for n in range(I):
            gate[e, n, rng.choice(H, 8, replace=False)] = 1
    up = rng.choice([-1, 1], (El, I, H))
    for e in range(El):
        for n in range(I):
            up[e, n, rng.choice(H, H // 2, replace=False)] = 0
    w13v = np.concatenate([gate, up], 1)
    s13 = np.empty((El, 2 * I // 128, H // 128), np.float32)
    s13[:, : I // 128] = 0.5
    s13[:, I // 128:] = np.exp2(rng.integers(-2, 0, (El, I // 128, H // 128)))
    logits, bias, _ = W.gen_router(cfg, seed, device="cuda")
    # w2 of the usual recipe, its scales times 2^-12 (exact) so that the outputs
    # are of order one, like the workloads' the plain tolerance is stated for
    # (the intermediate here is of order 10^4)
    base = W.generate(cfg.with_(T=1), seed, device="cuda")
    inp = W.MoEInputs(cfg, seed, torch.from_numpy(codes[xv + 16]).cuda(), torch.from_numpy(sx).cuda(),
                      logits, bias, torch.from_numpy(codes[w13v + 16]).cuda(), torch.from_numpy(s13).cuda(),
                      base.w2, base.w2_scale * 2.0 ** -12, base.hot)
    return inp, xv, sx, w13v, s13


def _requant(a):
    ab = a.reshape(-1, 128)
    amax = np.abs(ab).max(1)
    scale = np.where(amax > 0, (amax / np.float32(448.0)).astype(np.float32), np.float32(1.0))
    q = torch.from_numpy((ab / scale[:, None]).astype(np.float32)).clamp(-448, 448).to(torch.float8_e4m3fn)
    return q.view(torch.uint8).numpy().reshape(a.shape), scale.astype(np.float32).reshape(a.shape[0], -1)


# rows per expert T*k/E_g = 2 (gate/up-split narrow GEMM1), 8 (narrow), 32
# (32-row LDS kernel), 80 / 160 / 400 (64-, 128-, 256-row tile kernels)
@pytest.mark.parametrize("T", [8, 32, 128, 320, 640, 1600])
def test_exact_integer_intermediate(M, T):
    cfg = BASE.with_(T=T)
    log(f"exact T={T}")
    inp, xv, sx, w13v, s13 = exact_inputs(cfg, T)
    s = M.Shape.of(cfg)
    ro = M.alloc_route_out(s)
    ws = M.alloc_workspace(s)
    M.fused_fp8(s, inp.hidden, inp.hidden_scale, inp.logits, inp.bias, inp.w13, inp.w13_scale,
                inp.w2, inp.w2_scale, route_out=ro, workspace=ws)
    torch.cuda.synchronize()
    ref = oracle_route(cfg, inp)
    offs, perm = ref["expert_offsets"], ref["perm_token"]
    P = int(offs[-1])
    act, act_s = M.debug_act_views(s, ws)
    act, act_s = act[:P].cpu().numpy(), act_s[:P].cpu().numpy()
    I = cfg.I
    for e in range(cfg.num_local_experts):
        rows = np.arange(offs[e], offs[e + 1])
        if not rows.size:
            continue
        toks = perm[rows]
        # GEMM1 as an int64 product of the integer codes times the power-of-two scales
        xs = (xv[toks] * np.repeat(sx[toks], 128, 1)).astype(np.float64)
        ws_full = np.repeat(np.repeat(s13[e], 128, 0), 128, 1).astype(np.float64)
        g = xs @ (w13v[e] * ws_full).T
        assert (g[:, :I] >= 20).all() and (np.abs(g[:, :I] * g[:, I:]) <= 2.0 ** 20).all()
        a = (g[:, :I] * g[:, I:]).astype(np.float32)
        assert (a.astype(np.float64) == g[:, :I] * g[:, I:]).all()
        q, qs = _requant(a)
        assert (act[rows] == q).all(), f"expert {e}: {(act[rows] != q).sum()} codes differ"
        assert (act_s[rows].view(np.int32) == qs.view(np.int32)).all(), f"expert {e}: scales differ"
    stats = layer_parity(M, cfg, inp, what=f"exact T={T}")
    assert stats["flips"] == 0 and stats["scale_diffs"] == 0 and stats["beyond_plain_tol"] == 0
