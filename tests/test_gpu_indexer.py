"""GPU parity of the DSA TopK indexer (paper Section 3.1.3) through the C-ABI,
against the CPU oracle.

Scores follow one fixed fp32 sequence on both sides and must match bit for
bit; the returned indices (physical cache indices of each sequence's TopK
tokens, ascending position order, padded with -1) must match exactly."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def M():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_14560_amd as M
    M.lib()  # raises if the library is not built
    return M


def _host(x):
    return (x.q.cpu().numpy(), x.weights.cpu().numpy(), x.k_cache.cpu().numpy(),
            x.k_scale.cpu().numpy(), x.block_table.cpu().numpy(), x.seq_lens.cpu().numpy())


def _dev(x):
    return (x.q, x.weights, x.k_cache, x.k_scale, x.block_table, x.seq_lens)


@pytest.mark.parametrize("name", ["dsa_small", "dsa_paper_long", "dsa_short"])
def test_dsa_scores_bitexact(M, name):
    cfg = W.INDEXER_CONFIGS[name]
    log(f"dsa scores {name}")
    x = W.generate_indexer(cfg, 1, device="cuda")
    got = M.dsa_debug_scores(*_dev(x)).cpu().numpy()
    h = _host(x)
    for b, L in enumerate(cfg.seq_lens):
        ref = oracle.dsa_scores(*h, b)
        diff = got[b, :L].view(np.uint32) != ref.view(np.uint32)
        assert not diff.any(), f"b={b}: {diff.sum()} of {L} differ"


@pytest.mark.parametrize("name,seed", [("dsa_small", 0), ("dsa_small", 1), ("dsa_paper_long", 0),
                                       ("dsa_short", 0), ("dsa_long", 0)])
def test_dsa_topk_exact(M, name, seed):
    """Sequences below, at and just past TopK, ragged last pages, an empty
    sequence, and long ones (up to 65,536 tokens) far past it."""
    cfg = W.INDEXER_CONFIGS[name]
    log(f"dsa topk {name} seed {seed}")
    x = W.generate_indexer(cfg, seed, device="cuda")
    got = M.dsa_topk_indexer(*_dev(x), topk=cfg.topk).cpu().numpy()
    ref = oracle.dsa_topk(*_host(x), cfg.topk)
    for b in range(cfg.B):
        assert (got[b] == ref[b]).all(), f"b={b} (seq_len {cfg.seq_lens[b]}): {(got[b] != ref[b]).sum()} differ"


@pytest.mark.parametrize("ps", [8, 16, 1])
def test_dsa_topk_page_sizes(M, ps):
    """Pages smaller than, equal to and far below a select thread's 16
    consecutive positions (several pages per thread), against the oracle."""
    cfg = W.IndexerConfig(f"ps{ps}", (700, 300, 2000, 5000), page_size=ps, topk=512)
    log(f"dsa topk page size {ps}")
    x = W.generate_indexer(cfg, 6, device="cuda")
    got = M.dsa_topk_indexer(*_dev(x), topk=cfg.topk).cpu().numpy()
    ref = oracle.dsa_topk(*_host(x), cfg.topk)
    for b in range(cfg.B):
        assert (got[b] == ref[b]).all(), f"b={b}: {(got[b] != ref[b]).sum()} differ"


@pytest.mark.parametrize("cfg", [W.IndexerConfig("ties", (3000, 5000, 300), topk=512),
                                 # block tables of 16,384+ tokens: the slice-parallel compaction,
                                 # equal keys spread over many 2,048-position slices
                                 W.IndexerConfig("ties_wide", (20000, 17000, 300), topk=4096)],
                         ids=lambda c: c.name)
def test_dsa_topk_ties(M, cfg):
    """Keys and queries from a handful of values with equal weights: many exactly
    equal scores straddle the TopK threshold, and the lower positions must win."""
    x = W.generate_indexer(cfg, 2, device="cuda")
    g = torch.Generator(device="cpu").manual_seed(3)
    bits = lambda shape: torch.randint(0, 2, shape, generator=g).float().to(torch.float8_e4m3fn).view(torch.uint8)
    q = bits(tuple(x.q.shape))
    q[:, 1:, :] = 0  # one live head: every score is 0.5 * (a count of at most 128)
    x.q = q.cuda()
    x.k_cache = bits(tuple(x.k_cache.shape)).cuda()
    x.k_scale = torch.ones_like(x.k_scale)
    x.weights = torch.full_like(x.weights, 0.5)
    got = M.dsa_topk_indexer(*_dev(x), topk=cfg.topk).cpu().numpy()
    h = _host(x)
    sc = oracle.dsa_scores(*h, 1)
    thr = np.sort(sc)[::-1][cfg.topk - 1]
    log(f"ties: {(sc == thr).sum()} scores equal the threshold score")
    assert (sc == thr).sum() > 10
    ref = oracle.dsa_topk(*h, cfg.topk)
    assert (got == ref).all()


def test_dsa_topk_above_every_length_wide(M):
    """A block table of 16,384 tokens with TopK above every sequence length: every
    token in position order, then -1 up to TopK (past the block table's length)."""
    cfg = W.IndexerConfig("wide_short", (16384, 9000, 100, 0), topk=20000)
    x = W.generate_indexer(cfg, 8, device="cuda")
    got = M.dsa_topk_indexer(*_dev(x), topk=cfg.topk).cpu().numpy()
    ref = oracle.dsa_topk(*_host(x), cfg.topk)
    assert (got == ref).all()


def test_dsa_out_of_range_device_inputs(M):
    """Sequence lengths beyond the block table and negative ones are clamped on the
    device (no fault): they act as the longest and the empty sequence."""
    cfg = W.IndexerConfig("clamp", (700, 700, 300), topk=256)
    x = W.generate_indexer(cfg, 4, device="cuda")
    ref = oracle.dsa_topk(*_host(x), cfg.topk)
    x.seq_lens = torch.tensor([700, 10 ** 6, -5], dtype=torch.int32, device="cuda")
    got = M.dsa_topk_indexer(*_dev(x), topk=cfg.topk).cpu().numpy()
    assert (got[0] == ref[0]).all()
    h = list(_host(x))
    h[5] = np.array([700, cfg.max_pages * cfg.page_size, 0], np.int32)
    ref2 = oracle.dsa_topk(*h, cfg.topk)
    assert (got[1] == ref2[1]).all()    # as long as the block table allows
    assert (got[2] == -1).all()         # empty


def test_dsa_deterministic(M):
    cfg = W.INDEXER_CONFIGS["dsa_paper_long"]
    x = W.generate_indexer(cfg, 5, device="cuda")
    a = M.dsa_topk_indexer(*_dev(x), topk=cfg.topk)
    b = M.dsa_topk_indexer(*_dev(x), topk=cfg.topk)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
