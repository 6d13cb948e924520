"""GPU parity of the HIP path (through the C-ABI) against the CPU oracle.

Routing, permutation and the FP8 encoder must match bit for bit.  The
re-quantised FP8 intermediate must lie in the oracle's admissible set with
few flips, and the bf16 output must satisfy |gpu - ref| <= 1e-2 + 2e-2 |ref|
on every element, widened only by the oracle's bound on what the observed
intermediate differences can move (gpu_helpers.layer_parity).  GEMM2 and the
combine are also checked alone on the oracle's intermediate with the plain
tolerance.  Full-size configurations compare every token's routing and, where
the oracle would take minutes, a sample of output rows (tokens are
independent, so a sampled row is exact)."""
import numpy as np
import pytest
import torch

import gfx950_mfma_model as mm
import oracle
import workloads as W
from gpu_helpers import (assert_out_close, check_route, inputs, layer_parity, log, oracle_forward,
                         oracle_route, run_fused)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def M():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_14560_amd as M
    M.lib()  # raises if the library is not built
    return M


# ------------------------------------------------------------ building blocks
def test_sigmoid_bitexact(M):
    bits_hi = np.float32(80.0).view(np.uint32)
    pos = np.arange(0, int(bits_hi) + 1, 29, dtype=np.uint32).view(np.float32)
    xs = np.concatenate([-pos[::-1], pos, np.float32([100.0, -100.0, 1e30, -1e30, 0.0, -0.0])])
    log(f"sigmoid: {xs.size} inputs")
    got = M.debug_sigmoid(torch.from_numpy(xs).cuda()).cpu().numpy()
    ref = oracle.sigmoid(xs)
    diff = got.view(np.uint32) != ref.view(np.uint32)
    assert not diff.any(), f"{diff.sum()} mismatches, e.g. x={xs[diff][:4]}"


def test_e4m3_encoder_bitexact(M):
    vals = np.array([oracle.e4m3_decode(c) for c in range(0x7F)], np.float64)
    mids = ((vals[:-1] + vals[1:]) / 2).astype(np.float32)
    xs = np.concatenate([mids, np.nextafter(mids, np.float32(np.inf)),
                         np.nextafter(mids, np.float32(0)), vals.astype(np.float32)])
    rng = np.random.default_rng(0)
    xs = np.concatenate([xs, -xs, (rng.standard_normal(1 << 20) * np.exp2(rng.uniform(-12, 9, 1 << 20))).astype(np.float32),
                         np.float32([448.0, 449.0, 470.0, 1e6, -1e6])])
    got = M.debug_e4m3_encode(torch.from_numpy(xs).cuda()).cpu().numpy()
    ref = oracle.e4m3_encode_array(xs)
    diff = got != ref
    assert not diff.any(), f"{diff.sum()} mismatches, e.g. x={xs[diff][:4]} gpu={got[diff][:4]} ref={ref[diff][:4]}"


def _e4m3_codes(rng, shape, kind):
    """Random e4m3 codes: every finite code uniformly, or the codes of
    block-quantised normal data (what the layer sees)."""
    if kind == "uniform":
        c = rng.integers(0, 256, size=shape).astype(np.uint8)
        c[(c & 0x7F) == 0x7F] = 0x38
        return c
    x = rng.standard_normal(shape).astype(np.float32)
    amax = np.abs(x).max(-1, keepdims=True)
    q = torch.from_numpy(x / (amax / 448.0)).clamp(-448, 448).to(torch.float8_e4m3fn)
    return q.view(torch.uint8).numpy()


@pytest.mark.parametrize("kind", ["quantised", "quantised_zeros", "subnormal_mix", "uniform"])
def test_mfma_block_within_bound(M, kind):
    """One FP8 matrix-core block product, as the GEMM kernels issue it, stays
    within the per-block error bound the oracle's admissible sets assume
    (2^(E_kb - 6) + 2^-19 sum |p|) of the exact sum, on block-quantised data
    (what GEMM1 sees), with zeros, with injected subnormals and on uniformly
    random codes.  Diagnostic, not gated: how often the diagnostic model of the
    matrix core (tests/gfx950_mfma_model.py) reproduces the result bit for bit."""
    rng = np.random.default_rng({"quantised": 1, "quantised_zeros": 2, "subnormal_mix": 3, "uniform": 0}[kind])
    n = 2048
    if kind == "uniform":
        a, b = _e4m3_codes(rng, (n, 16, 128), "uniform"), _e4m3_codes(rng, (n, 16, 128), "uniform")
    else:
        a, b = _e4m3_codes(rng, (n, 16, 128), "q"), _e4m3_codes(rng, (n, 16, 128), "q")
        if kind == "quantised_zeros":
            a[rng.random(a.shape) < 0.1] = 0
        if kind == "subnormal_mix":
            for X in (a, b):
                m = rng.random(X.shape) < 0.05
                X[m] = rng.integers(1, 8, size=m.sum()).astype(np.uint8)
    d = M.debug_mfma_block(torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()).cpu().numpy()
    A = np.broadcast_to(a[:, :, None, :], (n, 16, 16, 128))
    B = np.broadcast_to(b[:, None, :, :], (n, 16, 16, 128))
    exact = (mm.DEC[A] * mm.DEC[B]).sum(-1)
    err = np.abs(d.astype(np.float64) - exact)
    bound = mm.block_bound(A, B)
    assert (err <= bound).all(), f"{(err > bound).sum()} block sums beyond the bound"
    model = mm.block_dot(A, B)
    log(f"{kind}: max err/bound {float((err / bound).max()):.3g}; diagnostic model differs in "
        f"{int((model.view(np.uint32) != d.view(np.uint32)).sum())} of {d.size} block sums")


# ------------------------------------------------------------ routing
ROUTE_CASES = [("tiny", 0), ("tiny", 1), ("small_ragged", 0), ("small_dense", 0), ("small_g6", 0), ("small_many", 0),
               ("small_many", 3), ("decode", 0), ("decode", 1), ("decode", 2), ("mid", 0), ("mid", 1),
               ("small_t64", 0), ("small_t128", 0), ("small_t256", 0), ("prefill", 0), ("skewed", 0),
               ("median", 0), ("long", 0)]


@pytest.mark.parametrize("name,seed", ROUTE_CASES)
def test_route_bitexact(M, name, seed):
    cfg = W.all_configs()[name]
    log(f"route {name} seed {seed}")
    logits, bias, _ = W.gen_router(cfg, seed, device="cuda")
    s = M.Shape.of(cfg)
    ro = M.route(s, logits, bias)
    torch.cuda.synchronize()
    ref_ids, ref_w = oracle.route(oracle.shape_of(cfg), logits.cpu().numpy(), bias.cpu().numpy())
    offs, perm, pr = oracle.permute(oracle.shape_of(cfg), ref_ids)
    check_route(cfg, ro, dict(topk_ids=ref_ids, topk_weights=ref_w, expert_offsets=offs,
                              perm_token=perm, pair_row=pr))


@pytest.mark.parametrize("T", [1, 31, 32, 33, 255, 256, 257])
def test_route_batch_sizes(M, T):
    """Routing and permutation at batch sizes around a wave of tokens and the
    256-token permutation chunk (one chunk, one chunk full, two chunks), bit
    for bit."""
    cfg = W.CONFIGS["decode"].with_(T=T)
    logits, bias, _ = W.gen_router(cfg, 7, device="cuda")
    ro = M.route(M.Shape.of(cfg), logits, bias)
    torch.cuda.synchronize()
    ref_ids, ref_w = oracle.route(oracle.shape_of(cfg), logits.cpu().numpy(), bias.cpu().numpy())
    offs, perm, pr = oracle.permute(oracle.shape_of(cfg), ref_ids)
    check_route(cfg, ro, dict(topk_ids=ref_ids, topk_weights=ref_w, expert_offsets=offs,
                              perm_token=perm, pair_row=pr))


def test_route_ties_bitexact(M):
    """Logits on a coarse grid and zero bias produce many exactly equal keys; the
    lower expert / group index must win every tie."""
    cfg = W.CONFIGS["decode"].with_(T=512)
    g = torch.Generator().manual_seed(5)
    logits = (torch.randn(cfg.T, cfg.num_experts, generator=g) * 2).round() / 2
    bias = torch.zeros(cfg.num_experts)
    bias[::3] = 0.25
    ro = M.route(M.Shape.of(cfg), logits.cuda(), bias.cuda())
    torch.cuda.synchronize()
    ref_ids, ref_w = oracle.route(oracle.shape_of(cfg), logits.numpy(), bias.numpy())
    offs, perm, pr = oracle.permute(oracle.shape_of(cfg), ref_ids)
    check_route(cfg, ro, dict(topk_ids=ref_ids, topk_weights=ref_w, expert_offsets=offs,
                              perm_token=perm, pair_row=pr))


# ------------------------------------------------------------ whole layer
FULL_CASES = [("tiny", 0), ("small_ragged", 0), ("small_ragged", 1), ("small_dense", 0), ("small_g6", 0),
              ("small_many", 0), ("small_t64", 0), ("small_t64", 1), ("small_t128", 0), ("small_t128", 2),
              ("small_t256", 0), ("small_t256_h640", 0), ("small_decode_all", 0), ("small_wide_i", 0),
              ("decode", 0),
              ("decode", 1), ("mid", 0), ("median", 0)]


@pytest.mark.parametrize("name,seed", FULL_CASES)
def test_fused_full_parity(M, name, seed):
    cfg = W.all_configs()[name]
    log(f"fused {name} seed {seed}: generating")
    layer_parity(M, cfg, inputs(cfg, seed), what=f"{name}/{seed}")


def test_fused_prefill_full_parity(M):
    """T = 4096 (32 of 256 experts resident): every token's output."""
    cfg = W.CONFIGS["prefill"]
    log("fused prefill: generating")
    layer_parity(M, cfg, inputs(cfg, 0), what="prefill")


def _sample_tokens(cfg, ref, n, seed=0):
    """Random tokens, plus the first and last rows of the two busiest experts and
    a token with the most resident experts."""
    rng = np.random.default_rng(seed)
    toks = set(rng.choice(cfg.T, size=min(n, cfg.T), replace=False).tolist())
    offs, perm = ref["expert_offsets"], ref["perm_token"]
    counts = np.diff(offs)
    for e in np.argsort(-counts)[:2]:
        if counts[e]:
            toks.update([int(perm[offs[e]]), int(perm[offs[e + 1] - 1])])
    nloc = (ref["pair_row"] >= 0).sum(1)
    toks.add(int(np.argmax(nloc)))
    return np.array(sorted(toks), np.int32)


@pytest.mark.parametrize("name,n", [("skewed", 24), ("long", 32)])
def test_fused_sampled_parity(M, name, n):
    cfg = W.CONFIGS[name]
    log(f"fused {name}: generating")
    inp = inputs(cfg, 0)
    toks = _sample_tokens(cfg, oracle_route(cfg, inp), n)
    layer_parity(M, cfg, inp, tokens=toks, what=name)


@pytest.mark.parametrize("r", range(8))
def test_expert_slice_offsets(M, r):
    """Each of the 8 slices of 32 experts (one per routing group) as the resident set."""
    cfg = W.CONFIGS["decode"].with_(T=48, local_expert_offset=32 * r)
    log(f"slice {r}")
    layer_parity(M, cfg, inputs(cfg, 11), staged=False, what=f"slice {r}")


def test_single_token(M):
    cfg = W.CONFIGS["decode"].with_(T=1, local_expert_offset=0)
    for seed in range(4):
        layer_parity(M, cfg, inputs(cfg, seed), what=f"T=1 seed {seed}")


def test_no_resident_pairs(M):
    """A bias that keeps every token away from the resident group: P = 0 and the
    output is exactly zero."""
    cfg = W.all_configs()["small_ragged"].with_(local_expert_offset=0, num_local_experts=8)
    inp = inputs(cfg, 2)
    bias = inp.bias.clone()
    bias[:8] -= 50.0
    inp2 = W.MoEInputs(**{**inp.__dict__, "bias": bias})
    out, ro, _ = run_fused(M, cfg, inp2)
    assert int(ro["expert_offsets"][-1]) == 0
    assert (ro["pair_row"] == -1).all()
    assert (out == 0).all()


def test_one_expert_takes_all(M):
    """One expert chosen by every token (a single M-tile list covering all rows)."""
    cfg = W.all_configs()["small_many"]
    inp = inputs(cfg, 4)
    bias = inp.bias.clone()
    bias[5] += 50.0
    inp2 = W.MoEInputs(**{**inp.__dict__, "bias": bias})
    ref = oracle_route(cfg, inp2)
    assert np.diff(ref["expert_offsets"])[5] == cfg.T
    layer_parity(M, cfg, inp2, what="one expert takes all")


def test_empty_batch(M):
    cfg = W.CONFIGS["decode"].with_(T=0)
    s = M.Shape.of(cfg)
    inp = inputs(W.CONFIGS["decode"].with_(T=1), 0)
    out = torch.empty(0, cfg.H, dtype=torch.bfloat16, device="cuda")
    M.fused_fp8(s, inp.hidden[:0], inp.hidden_scale[:0], inp.logits[:0], inp.bias, inp.w13,
                inp.w13_scale, inp.w2, inp.w2_scale, out=out, workspace=M.alloc_workspace(s))
    ro = M.route(s, inp.logits[:0], inp.bias)
    torch.cuda.synchronize()
    assert (ro["expert_offsets"] == 0).all()


def test_deterministic(M):
    cfg = W.CONFIGS["decode"]
    inp = inputs(cfg, 0)
    out1, ro1, _ = run_fused(M, cfg, inp)
    out2, ro2, _ = run_fused(M, cfg, inp)
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    P = int(ro1["expert_offsets"][-1])
    for k in ro1:
        n = P if k == "perm_token" else None
        assert torch.equal(ro1[k][:n], ro2[k][:n]), k


def test_staged_events(M):
    cfg = W.CONFIGS["decode"]
    inp = inputs(cfg, 0)
    s = M.Shape.of(cfg)
    ws = M.alloc_workspace(s)
    out = torch.empty(cfg.T, cfg.H, dtype=torch.bfloat16, device="cuda")
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(M.num_stages() + 1)]
    M.fused_fp8_staged(s, inp.hidden, inp.hidden_scale, inp.logits, inp.bias, inp.w13,
                       inp.w13_scale, inp.w2, inp.w2_scale, out, ws, evs)
    torch.cuda.synchronize()
    ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(M.num_stages())]
    log(f"stage ms: {dict(zip(M.stage_names(), ms))}")
    assert all(m >= 0 for m in ms)
    out2, _, _ = run_fused(M, cfg, inp)
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))
