"""GPU parity of the router projection path (stage (1)'s linear projection on
the device) through the C-ABI, against the CPU oracle.

The logits follow one fixed fp32 sequence on both sides, so they must match
bit for bit; so must the expert choice, the routing weights and the
permutation that follow.  The whole layer with the projection must give the
same bf16 output as the layer fed the oracle's logits (bit for bit: identical
logits, identical path after them) and stay within the output tolerance of
the oracle.  Full-size batches are compared on sampled tokens (the projection
of a token depends on that token's row only)."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import inputs, layer_parity, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def M():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_14560_amd as M
    M.lib()  # raises if the library is not built
    return M


def _router_inputs(cfg, seed):
    hq, hs = W.gen_hidden(cfg, seed, device="cuda")
    wg = W.gen_router_weight(cfg, seed, device="cuda")
    _, bias, _ = W.gen_router(cfg.with_(T=1), seed, device="cuda")
    return hq, hs, wg, bias


def _oracle_logits(cfg, hq, hs, wg, tokens=None):
    h, s = hq.cpu().numpy(), hs.cpu().numpy()
    if tokens is not None:
        h, s = h[tokens], s[tokens]
    shape = oracle.shape_of(cfg.with_(T=h.shape[0]))
    return oracle.router_logits(shape, h, s, wg.cpu().numpy())


def _assert_bits(got, ref, what):
    diff = got.view(np.uint32) != ref.view(np.uint32)
    assert not diff.any(), f"{what}: {diff.sum()} of {diff.size} differ, first at {np.argwhere(diff)[:4].tolist()}"


LOGIT_CASES = [("tiny", 8), ("small_ragged", 77), ("small_g6", 50), ("small_many", 300),
               ("decode", 1), ("decode", 16), ("decode", 33), ("decode", 256), ("decode", 600)]


@pytest.mark.parametrize("name,T", LOGIT_CASES)
def test_router_logits_bitexact(M, name, T):
    """Token counts around the projection's 16-token tiles (1, 16, 33) and its
    32-token tiles for large batches (600: a ragged last tile), expert counts
    below and across its 64-expert tiles (16, 32, 64, 96, 256)."""
    cfg = W.all_configs()[name].with_(T=T)
    log(f"router logits {name} T={T}")
    hq, hs, wg, _ = _router_inputs(cfg, 3)
    got = M.debug_router_logits(M.Shape.of(cfg), hq, hs, wg)
    torch.cuda.synchronize()
    _assert_bits(got.cpu().numpy(), _oracle_logits(cfg, hq, hs, wg), "logits")


def test_router_logits_exact_integers(M):
    """Integer codes, small integer weights, power-of-two scales: every partial
    sum is exact, so the logits equal an integer matrix product (checked on
    the device result directly, not through the oracle)."""
    cfg = W.CONFIGS["decode"].with_(T=20)
    g = torch.Generator().manual_seed(9)
    xv = torch.randint(-16, 17, (cfg.T, cfg.H), generator=g)
    wv = torch.randint(-8, 9, (cfg.num_experts, cfg.H), generator=g)
    xs = torch.exp2(torch.randint(-4, 3, (cfg.T, cfg.H // 128), generator=g).float())
    hq = xv.float().to(torch.float8_e4m3fn).view(torch.uint8)
    got = M.debug_router_logits(M.Shape.of(cfg), hq.cuda(), xs.cuda(), wv.float().cuda())
    torch.cuda.synchronize()
    ref = torch.einsum("tbi,ebi->te", (xv.double().reshape(cfg.T, -1, 128) * xs.double()[:, :, None]),
                       wv.double().reshape(cfg.num_experts, -1, 128))
    assert (got.cpu().double() == ref).all()


ROUTE_CASES = [("tiny", 0), ("small_ragged", 0), ("small_g6", 0), ("small_many", 1), ("decode", 0),
               ("decode", 1), ("mid", 0)]


@pytest.mark.parametrize("name,seed", ROUTE_CASES)
def test_route_hidden_bitexact(M, name, seed):
    cfg = W.all_configs()[name]
    log(f"route_hidden {name} seed {seed}")
    hq, hs, wg, bias = _router_inputs(cfg, seed)
    s = M.Shape.of(cfg)
    ro = M.route_hidden(s, hq, hs, wg, bias)
    torch.cuda.synchronize()
    os_ = oracle.shape_of(cfg)
    ids, w = oracle.route(os_, _oracle_logits(cfg, hq, hs, wg), bias.cpu().numpy())
    offs, perm, pr = oracle.permute(os_, ids)
    assert (ro["topk_ids"].cpu().numpy() == ids).all()
    _assert_bits(ro["topk_weights"].cpu().numpy(), w, "topk_weights")
    assert (ro["expert_offsets"].cpu().numpy() == offs).all()
    P = int(offs[-1])
    assert (ro["perm_token"].cpu().numpy()[:P] == perm).all()
    assert (ro["pair_row"].cpu().numpy() == pr).all()


@pytest.mark.parametrize("name", ["prefill", "skewed"])
def test_route_hidden_sampled_full_size(M, name):
    """Full-size batches in the launch configuration of the layer: the logits and
    expert choice of sampled tokens (first, last, random) bit for bit."""
    cfg = W.CONFIGS[name]
    log(f"route_hidden sampled {name}")
    hq, hs, wg, bias = _router_inputs(cfg, 0)
    s = M.Shape.of(cfg)
    ws = M.alloc_workspace(s)
    ro = M.route_hidden(s, hq, hs, wg, bias, workspace=ws)
    lg = M.debug_router_logits(s, hq, hs, wg, workspace=ws)
    torch.cuda.synchronize()
    rng = np.random.default_rng(4)
    toks = np.unique(np.concatenate([[0, 15, 16, cfg.T - 1], rng.choice(cfg.T, 60, replace=False)]))
    ref = _oracle_logits(cfg, hq, hs, wg, toks)
    _assert_bits(lg.cpu().numpy()[toks], ref, "logits")
    ids, w = oracle.route(oracle.shape_of(cfg.with_(T=len(toks))), ref, bias.cpu().numpy())
    assert (ro["topk_ids"].cpu().numpy()[toks] == ids).all()
    _assert_bits(ro["topk_weights"].cpu().numpy()[toks], w, "topk_weights")


@pytest.mark.parametrize("name,seed", [("tiny", 0), ("small_ragged", 1), ("small_t64", 0), ("decode", 0)])
def test_fused_router_matches_fused_with_oracle_logits(M, name, seed):
    """The layer with the projection equals, bit for bit, the layer fed the
    oracle's logits; on the small cases also within tolerance of the oracle."""
    cfg = W.all_configs()[name]
    log(f"fused_router {name} seed {seed}")
    inp = inputs(cfg, seed)
    wg = W.gen_router_weight(cfg, seed, device="cuda")
    s = M.Shape.of(cfg)
    ro = M.alloc_route_out(s)
    out_r = M.fused_fp8_router(s, inp.hidden, inp.hidden_scale, wg, inp.bias, inp.w13,
                               inp.w13_scale, inp.w2, inp.w2_scale, route_out=ro)
    lg = torch.from_numpy(_oracle_logits(cfg, inp.hidden, inp.hidden_scale, wg)).cuda()
    out_l = M.fused_fp8(s, inp.hidden, inp.hidden_scale, lg, inp.bias, inp.w13, inp.w13_scale,
                        inp.w2, inp.w2_scale)
    torch.cuda.synchronize()
    assert torch.equal(out_r.view(torch.int16), out_l.view(torch.int16))
    if name != "decode":
        # the layer fed those logits (bit-identical to out_r) against the oracle
        inp_o = W.MoEInputs(**{**inp.__dict__, "logits": lg})
        layer_parity(M, cfg, inp_o, staged=False, what=f"fused_router {name}/{seed}")


def test_route_hidden_empty_batch(M):
    cfg = W.CONFIGS["decode"].with_(T=0)
    s = M.Shape.of(cfg)
    hq, hs, wg, bias = _router_inputs(cfg.with_(T=1), 0)
    ro = M.alloc_route_out(s)
    ro["expert_offsets"].fill_(7)
    M.route_hidden(s, hq[:0], hs[:0], wg, bias, route_out=ro)
    torch.cuda.synchronize()
    assert (ro["expert_offsets"].cpu() == 0).all()
