"""GPU parity of the HIP path (through the C-ABI) against the CPU oracle.

Routing, permutation and the FP8 encoder must match bit for bit; the bf16
output must satisfy |gpu - ref| <= 1e-2 + 2e-2 |ref| on every element (ref =
the oracle's bf16 output).  Full-size configurations compare every token's
routing and a sample of output rows (tokens are independent, so a sampled row
is exact)."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import assert_out_close, experts_of, inputs, log, oracle_forward, oracle_route

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def M():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_14560_amd as M
    M.lib()  # raises if the library is not built
    return M


def run_fused(M, cfg, inp, route=True):
    s = M.Shape.of(cfg)
    ro = M.alloc_route_out(s) if route else None
    ws = M.alloc_workspace(s)
    out = M.fused_fp8(s, inp.hidden, inp.hidden_scale, inp.logits, inp.bias, inp.w13,
                      inp.w13_scale, inp.w2, inp.w2_scale, route_out=ro, workspace=ws)
    torch.cuda.synchronize()
    return out, ro, ws


def check_route(cfg, ro, ref):
    ids = ro["topk_ids"].cpu().numpy()
    assert (ids == ref["topk_ids"]).all(), f"topk_ids differ at {np.argwhere(ids != ref['topk_ids'])[:5]}"
    w = ro["topk_weights"].cpu().numpy()
    assert (w.view(np.int32) == ref["topk_weights"].view(np.int32)).all(), "topk_weights differ"
    offs = ro["expert_offsets"].cpu().numpy()
    assert (offs == ref["expert_offsets"]).all(), "expert_offsets differ"
    P = int(offs[-1])
    assert (ro["perm_token"].cpu().numpy()[:P] == ref["perm_token"]).all(), "perm_token differs"
    assert (ro["pair_row"].cpu().numpy() == ref["pair_row"]).all(), "pair_row differs"


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
def test_mfma_block_rule(M, kind):
    """The FP8 block product that GEMM1 promotes, against the oracle's statement
    of the matrix cores' block arithmetic (groups of 8 products truncated to the
    group exponent's 2^-13 grid, group sums added in order in fp32).  Block-
    quantised data -- what GEMM1 sees -- must match bit for bit.  The rule's
    known limit is partial sums that do not fit fp32 (a group exponent spread
    beyond 7 binades): the cross-group rounding then differs by an ulp in a few
    results, measured here on injected subnormals and on uniformly random codes."""
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
    ref = oracle.fp8_block_dot(np.broadcast_to(a[:, :, None, :], (n, 16, 16, 128)),
                               np.broadcast_to(b[:, None, :, :], (n, 16, 16, 128)))
    mism = d.view(np.uint32) != ref.view(np.uint32)
    log(f"{kind}: {mism.sum()} of {mism.size} block sums differ from the rule")
    if kind in ("quantised", "quantised_zeros"):
        assert not mism.any()
    elif kind == "subnormal_mix":
        ulps = np.abs(d.view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64))
        assert mism.mean() < 1e-3 and (ulps[mism] <= 4).all()
    else:
        assert mism.mean() < 0.25


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
              ("small_many", 0), ("small_t64", 0), ("small_t64", 1), ("small_t128", 0), ("small_t128", 2), ("small_t256", 0),
              ("decode", 0), ("decode", 1), ("mid", 0), ("median", 0)]


@pytest.mark.parametrize("name,seed", FULL_CASES)
def test_fused_full_parity(M, name, seed):
    cfg = W.all_configs()[name]
    log(f"fused {name} seed {seed}: generating")
    inp = inputs(cfg, seed)
    out, ro, _ = run_fused(M, cfg, inp)
    ref = oracle_route(cfg, inp)
    check_route(cfg, ro, ref)
    log(f"fused {name}: P={int(ref['expert_offsets'][-1])}, oracle running")
    ref_out, _, _ = oracle_forward(cfg, inp, ref_ids=ref["topk_ids"])
    err, mag = assert_out_close(out, ref_out, f"{name}/{seed}")
    log(f"fused {name}: max |err| {err:.3g} (max |ref| {mag:.3g})")


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


@pytest.mark.parametrize("name,n", [("prefill", 40), ("skewed", 16), ("long", 24)])
def test_fused_sampled_parity(M, name, n):
    cfg = W.CONFIGS[name]
    log(f"fused {name}: generating")
    inp = inputs(cfg, 0)
    out, ro, _ = run_fused(M, cfg, inp)
    ref = oracle_route(cfg, inp)
    check_route(cfg, ro, ref)
    toks = _sample_tokens(cfg, ref, n)
    log(f"fused {name}: P={int(ref['expert_offsets'][-1])}, oracle on {len(toks)} tokens, "
        f"{len(experts_of(cfg, ref['topk_ids'], toks))} experts")
    ref_out, _, _ = oracle_forward(cfg, inp, tokens=toks, ref_ids=ref["topk_ids"])
    err, mag = assert_out_close(out[torch.from_numpy(toks).long().cuda()], ref_out, name)
    log(f"fused {name}: max |err| {err:.3g} (max |ref| {mag:.3g})")
    # rows of tokens without a resident expert are exactly zero
    none = np.flatnonzero((ref["pair_row"] < 0).all(1))
    if none.size:
        assert (out[torch.from_numpy(none).long().cuda()] == 0).all()


@pytest.mark.parametrize("r", range(8))
def test_expert_slice_offsets(M, r):
    """Each of the 8 slices of 32 experts (one per routing group) as the resident set."""
    cfg = W.CONFIGS["decode"].with_(T=48, local_expert_offset=32 * r)
    log(f"slice {r}")
    inp = inputs(cfg, 11)
    out, ro, _ = run_fused(M, cfg, inp)
    ref = oracle_route(cfg, inp)
    check_route(cfg, ro, ref)
    ref_out, _, _ = oracle_forward(cfg, inp, ref_ids=ref["topk_ids"])
    assert_out_close(out, ref_out, f"slice {r}")


def test_single_token(M):
    cfg = W.CONFIGS["decode"].with_(T=1, local_expert_offset=0)
    for seed in range(4):
        inp = inputs(cfg, seed)
        out, ro, _ = run_fused(M, cfg, inp)
        ref = oracle_route(cfg, inp)
        check_route(cfg, ro, ref)
        ref_out, _, _ = oracle_forward(cfg, inp, ref_ids=ref["topk_ids"])
        assert_out_close(out, ref_out, f"T=1 seed {seed}")


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
    out, ro, _ = run_fused(M, cfg, inp2)
    ref = oracle_route(cfg, inp2)
    check_route(cfg, ro, ref)
    counts = np.diff(ref["expert_offsets"])
    assert counts[5] == cfg.T
    ref_out, _, _ = oracle_forward(cfg, inp2, ref_ids=ref["topk_ids"])
    assert_out_close(out, ref_out, "one expert takes all")


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


@pytest.mark.parametrize("name,sampled", [("tiny", False), ("decode", False), ("small_many", False),
                                          ("small_t64", False), ("small_t128", False),
                                          ("small_t256", False), ("prefill", True),
                                          ("skewed", True)])
def test_requantised_intermediate(M, name, sampled):
    """The FP8 intermediate (after SwiGLU and re-quantisation) against the
    oracle's codes and scales, bit for bit (the oracle takes this decision in
    the kernel's precision): every resident pair, or at full size the three
    busiest experts' first row, the rows either side of the 128- and 256-row
    M-tile boundaries and the last row."""
    cfg = W.all_configs()[name]
    inp = inputs(cfg, 0)
    out, ro, ws = run_fused(M, cfg, inp)
    ref = oracle_route(cfg, inp)
    act, act_scale = M.debug_act_views(M.Shape.of(cfg), ws)
    act, act_scale = act.cpu().numpy(), act_scale.cpu().numpy()
    offs, perm = ref["expert_offsets"], ref["perm_token"]
    h = W.host_arrays(inp, experts=[e for e in range(cfg.num_local_experts) if offs[e + 1] > offs[e]])
    busiest = set(np.argsort(-np.diff(offs))[:3].tolist())
    flips, total, scale_diff = 0, 0, 0
    for e in range(cfg.num_local_experts):
        rows = range(offs[e], offs[e + 1])
        if sampled:
            if e not in busiest or not len(rows):
                continue
            rows = sorted({rows[min(i, len(rows) - 1)] for i in (0, 127, 128, 255, 256)} | {rows[-1]})
        for row in rows:
            t = perm[row]
            _, _, q, qs = oracle.expert_ffn(h["hidden"][t], h["hidden_scale"][t], h["w13"][e],
                                            h["w13_scale"][e], h["w2"][e], h["w2_scale"][e])
            flips += int((act[row] != q).sum())
            total += q.size
            scale_diff += int((act_scale[row].view(np.int32) != qs.view(np.int32)).sum())
    log(f"{name}: {flips} code differences of {total}, {scale_diff} scale differences")
    assert flips == 0 and scale_diff == 0


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
    ref = oracle_forward(cfg, inp)[0]
    assert_out_close(out, ref, "staged")
