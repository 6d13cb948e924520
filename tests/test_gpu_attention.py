"""GPU parity of the DSA sparse attention (paper Section 3.1.2) through the
C-ABI, against the fp64 CPU oracle.

No integer decision follows from these floats, so the bound is a tolerance:
the bf16 output within 1e-2 + 2e-2 |ref| elementwise (the layer's bound; a
bf16 rounding of the output is 2^-9 relative, fp32 accumulation of 2048
terms far less) and the fp32 LSE within 1e-4 + 1e-6 |ref|."""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_helpers import log

pytestmark = pytest.mark.gpu

ATOL, RTOL = 1e-2, 2e-2


@pytest.fixture(scope="module")
def M():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_14560_amd as M
    M.lib()  # raises if the library is not built
    return M


def _host(x):
    b = lambda t: t.contiguous().cpu().view(torch.int16).numpy().view(np.uint16)
    return b(x.q_nope), b(x.q_pe), b(x.ckv), b(x.kpe), x.indices.cpu().numpy()


def _check(M, x, tokens=None):
    from oracle import dsa_attention as A
    out, lse = M.dsa_sparse_attention(x.q_nope, x.q_pe, x.ckv, x.kpe, x.indices, x.sm_scale)
    torch.cuda.synchronize()
    ref_o, ref_l = A.sparse_attention(*_host(x), x.sm_scale, tokens=tokens)
    got_o = out.float().cpu().numpy()
    got_l = lse.cpu().numpy()
    if tokens is not None:
        got_o, got_l = got_o[tokens], got_l[tokens]
    err = np.abs(got_o - ref_o)
    used = (err / (ATOL + RTOL * np.abs(ref_o))).max()
    log(f"  out: {used:.3f} of the bound used at most")
    assert used <= 1.0, f"out: max err {err.max():.3g}"
    fin = np.isfinite(ref_l)
    assert (np.isneginf(got_l) == ~fin).all()
    lerr = np.abs(got_l[fin] - ref_l[fin])
    assert (lerr <= 1e-4 + 1e-6 * np.abs(ref_l[fin])).all(), f"lse: max err {lerr.max():.3g}"
    return err.max(), lerr.max() if lerr.size else 0.0


@pytest.mark.parametrize("name,seed", [("attn_small", 0), ("attn_pad", 0), ("attn_one", 0), ("attn_two", 1),
                                       ("attn_long", 0)])
def test_sparse_attention_parity(M, name, seed):
    """TopK 256 and 2048, sequences shorter than TopK (padded index lists), a
    one-entry sequence, and the paper's long representative (8 tokens, 8462
    pages)."""
    cfg = W.ATTENTION_CONFIGS[name]
    log(f"attention {name} seed {seed}")
    x = W.generate_attention(cfg, seed, device="cuda")
    e, le = _check(M, x)
    log(f"attention {name}: max |err| out {e:.3g}, lse {le:.3g}")


@pytest.mark.parametrize("cfg", [
    # 32 heads (two head groups per token), TopK 100 (a ragged last split of 36 entries)
    W.AttentionConfig("h32_k100", (90, 5000, 100), num_heads=32, topk=100),
    # 128 heads (DeepSeek-V3.2 without head sharding): 8 head groups; T*H = 512 picks the
    # 8-column merge
    W.AttentionConfig("h128", (3000, 2048, 70, 9000), num_heads=128),
    # TopK 1 and 65 (one split; two splits with a single entry in the second)
    W.AttentionConfig("k1", (1, 500), topk=1),
    W.AttentionConfig("k65", (65, 64, 3000), topk=65),
    # 40 tokens of mixed lengths: 1,280 split workgroups, T*H = 640 (8-column merge)
    W.AttentionConfig("t40", tuple(int(v) for v in np.random.default_rng(7).integers(1, 9000, 40)), topk=512),
], ids=lambda c: c.name)
def test_sparse_attention_shapes(M, cfg):
    log(f"attention {cfg.name}: T={cfg.T} H={cfg.num_heads} topk={cfg.topk}")
    x = W.generate_attention(cfg, 11, device="cuda")
    e, le = _check(M, x)
    log(f"attention {cfg.name}: max |err| out {e:.3g}, lse {le:.3g}")


def test_sparse_attention_empty_batch(M):
    cfg = W.ATTENTION_CONFIGS["attn_two"]
    x = W.generate_attention(cfg, 0, device="cuda")
    out, lse = M.dsa_sparse_attention(x.q_nope[:0], x.q_pe[:0], x.ckv, x.kpe, x.indices[:0], x.sm_scale)
    torch.cuda.synchronize()
    assert out.shape == (0, 16, 512) and lse.shape == (0, 16)


def test_sparse_attention_invalid_indices(M):
    """Index entries past the cache or negative are absent; a token with none left
    gets out = 0 and lse = -inf."""
    cfg = W.AttentionConfig("inv", (500, 500, 500), topk=128)
    x = W.generate_attention(cfg, 2, device="cuda")
    idx = x.indices.clone()
    idx[0, ::3] = 10 ** 8          # past the cache
    idx[1, :] = -1                 # nothing
    idx[2, 5:] = -7
    x.indices = idx
    ref = x.indices.clone()
    ref[0, ::3] = -1               # what the oracle takes them as
    out, lse = M.dsa_sparse_attention(x.q_nope, x.q_pe, x.ckv, x.kpe, x.indices, x.sm_scale)
    torch.cuda.synchronize()
    x.indices = ref
    _check(M, x)
    assert (out[1].float() == 0).all() and torch.isneginf(lse[1]).all()


def test_sparse_attention_deterministic(M):
    cfg = W.ATTENTION_CONFIGS["attn_two"]
    x = W.generate_attention(cfg, 3, device="cuda")
    a = M.dsa_sparse_attention(x.q_nope, x.q_pe, x.ckv, x.kpe, x.indices, x.sm_scale)
    b = M.dsa_sparse_attention(x.q_nope, x.q_pe, x.ckv, x.kpe, x.indices, x.sm_scale)
    torch.cuda.synchronize()
    assert torch.equal(a[0].view(torch.int16), b[0].view(torch.int16)) and torch.equal(a[1], b[1])
