"""Seeded synthetic workloads for the fused FP8 MoE layer.

This module is shared by the tests, the benchmark and the smoke check.  It
holds the configuration registry and the input generators only: none of the
layer's arithmetic lives here.  The paper evaluates on the FlashInfer-Bench
Fused MoE workloads (DeepSeek-V3 shapes, Section 3.1.1 and the workload-regime
table of Section 3.2.1); those are not available, so these seeded inputs of the
same shapes stand in for them.

Recipe (all draws from ``torch.Generator`` objects on the target device, one
per (seed, tensor id, expert) sub-stream, so a single expert can be
regenerated alone):
  * router logits  fp32 N(0, 1)                       [T, E_g]        id 1
  * routing bias   fp32 N(0, 0.1); in the skewed case  [E_g]           id 2
    +2.0 on ``hot_experts`` experts drawn by randperm                 id 6
  * hidden         N(0, 1) quantised to e4m3fn per 1x128 block          id 3
                   with fp32 scale = amax / 448                       [T, H]
  * w13 (gate rows [0,I), up rows [I,2I)), w2: N(0, 0.02) quantised   id 4, 5
    per 128x128 block, fp32 scale = amax / 448
  * router weight  fp32 N(0, 1/H) [E_g, H] (for the router projection:  id 7
    with N(0, 1) hidden rows the projected logits are about N(0, 1),
    the distribution of the logits drawn directly)
Input quantisation uses torch's own float8_e4m3fn conversion (round to nearest
even) after clamping to +-448; an all-zero block gets scale 1.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np
import torch


@dataclass(frozen=True)
class MoEConfig:
    name: str
    T: int
    H: int
    I: int
    num_experts: int
    num_local_experts: int
    local_expert_offset: int
    n_group: int
    topk_group: int
    top_k: int
    routed_scaling_factor: float = 2.5
    hot_experts: int = 0
    hot_bias: float = 2.0

    def with_(self, **kw) -> "MoEConfig":
        return replace(self, **kw)


def _ds_v3(name: str, T: int, **kw) -> MoEConfig:
    base = dict(H=7168, I=2048, num_experts=256, num_local_experts=32,
                local_expert_offset=0, n_group=8, topk_group=4, top_k=8)
    base.update(kw)
    return MoEConfig(name=name, T=T, **base)


CONFIGS: dict[str, MoEConfig] = {
    # tiny case the oracle finishes in well under a second
    "tiny": MoEConfig("tiny", T=8, H=512, I=256, num_experts=16, num_local_experts=16,
                      local_expert_offset=0, n_group=4, topk_group=2, top_k=4),
    # DeepSeek-V3 shapes, 32 resident experts of a 256-expert router
    "decode": _ds_v3("decode", 16),
    "mid": _ds_v3("mid", 256),
    "prefill": _ds_v3("prefill", 4096),
    # all 256 experts resident, 16 hot experts
    "skewed": _ds_v3("skewed", 8192, num_local_experts=256, hot_experts=16),
    # context points at the paper's regime representatives: its median regime
    # (T = 64) and its longest workload (T = 14,107), same recipe as decode
    "median": _ds_v3("median", 64),
    "long": _ds_v3("long", 14107),
}

# Extra parity shapes: several tiles plus ragged tails, still fast on the CPU.
PARITY_CONFIGS: dict[str, MoEConfig] = {
    "small_ragged": MoEConfig("small_ragged", T=77, H=640, I=384, num_experts=32,
                              num_local_experts=12, local_expert_offset=8, n_group=4,
                              topk_group=2, top_k=6),
    "small_dense": MoEConfig("small_dense", T=40, H=256, I=256, num_experts=8,
                             num_local_experts=8, local_expert_offset=0, n_group=2,
                             topk_group=2, top_k=8),
    # a group count the routing kernel has no compile-time variant for
    "small_g6": MoEConfig("small_g6", T=50, H=256, I=256, num_experts=96,
                          num_local_experts=24, local_expert_offset=24, n_group=6,
                          topk_group=3, top_k=6),
    "small_many": MoEConfig("small_many", T=300, H=384, I=256, num_experts=64,
                            num_local_experts=64, local_expert_offset=0, n_group=8,
                            topk_group=4, top_k=8, hot_experts=4),
    # ~60 rows per expert: 64-row M-tiles; H = 384 leaves a 128-wide last
    # 256-column GEMM2 block, I = 256 a group of two column blocks
    "small_t64": MoEConfig("small_t64", T=160, H=384, I=256, num_experts=16,
                           num_local_experts=16, local_expert_offset=0, n_group=4,
                           topk_group=2, top_k=6),
    # ~128 rows per expert: 128-row M-tiles, 6 of 8 experts resident, three
    # intermediate blocks (I = 384), ragged GEMM2 columns (H = 640)
    "small_t128": MoEConfig("small_t128", T=256, H=640, I=384, num_experts=8,
                            num_local_experts=6, local_expert_offset=1, n_group=2,
                            topk_group=2, top_k=4),
    # 16 tokens, every expert resident: 128 pairs, more than the fused
    # GEMM2 + combine stages in LDS (its activation rows come from memory)
    "small_decode_all": MoEConfig("small_decode_all", T=16, H=1024, I=2048, num_experts=64,
                                  num_local_experts=64, local_expert_offset=0, n_group=8,
                                  topk_group=4, top_k=8),
    # 16 tokens with a wide intermediate (I = 8192): the fused GEMM2 + combine
    # would not fit its workgroup's LDS, so GEMM2 and the combine run apart
    "small_wide_i": MoEConfig("small_wide_i", T=16, H=256, I=8192, num_experts=16,
                              num_local_experts=16, local_expert_offset=0, n_group=4,
                              topk_group=4, top_k=8),
    # ~320 rows per expert with H = 640: 256-row tiles whose GEMM2 items take
    # the 256-column blocks in pairs, the last pair a single (ragged) block
    "small_t256_h640": MoEConfig("small_t256_h640", T=640, H=640, I=256, num_experts=8,
                                 num_local_experts=8, local_expert_offset=0, n_group=2,
                                 topk_group=2, top_k=4),
    # ~320 rows per expert: 256-row M-tiles with a ragged second tile
    "small_t256": MoEConfig("small_t256", T=640, H=384, I=256, num_experts=8,
                            num_local_experts=8, local_expert_offset=0, n_group=2,
                            topk_group=2, top_k=4),
}


def all_configs() -> dict[str, MoEConfig]:
    d = dict(CONFIGS)
    d.update(PARITY_CONFIGS)
    return d


# ---------------------------------------------------------------------------
# seeded sub-streams
# ---------------------------------------------------------------------------
TID_LOGITS, TID_BIAS, TID_HIDDEN, TID_W13, TID_W2, TID_HOT, TID_ROUTER_W = 1, 2, 3, 4, 5, 6, 7


def substream_seed(seed: int, tid: int, expert: int = 0) -> int:
    st = np.random.SeedSequence([int(seed), int(tid), int(expert)]).generate_state(2, np.uint32)
    return int((int(st[0]) << 31) ^ int(st[1])) & ((1 << 63) - 1)


def _gen(device, seed: int, tid: int, expert: int = 0) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(substream_seed(seed, tid, expert))
    return g


def quantize_blocks(x: torch.Tensor, br: int, bc: int):
    """Block quantisation used to synthesise inputs: (e4m3fn codes as uint8, fp32 scales)."""
    R, C = x.shape
    xb = x.reshape(R // br, br, C // bc, bc)
    amax = xb.abs().amax(dim=(1, 3))
    scale = torch.where(amax > 0, amax / 448.0, torch.ones_like(amax))
    q = (xb / scale[:, None, :, None]).clamp(-448.0, 448.0).to(torch.float8_e4m3fn)
    return q.reshape(R, C).view(torch.uint8), scale.to(torch.float32).contiguous()


def gen_router(cfg: MoEConfig, seed: int, device="cpu"):
    """(logits fp32 [T,E_g], bias fp32 [E_g], hot expert ids int64)."""
    logits = torch.randn(cfg.T, cfg.num_experts, generator=_gen(device, seed, TID_LOGITS),
                         device=device, dtype=torch.float32)
    bias = torch.randn(cfg.num_experts, generator=_gen(device, seed, TID_BIAS),
                       device=device, dtype=torch.float32) * 0.1
    hot = torch.empty(0, dtype=torch.int64)
    if cfg.hot_experts:
        g = torch.Generator(device="cpu")
        g.manual_seed(substream_seed(seed, TID_HOT))
        hot = torch.randperm(cfg.num_experts, generator=g)[: cfg.hot_experts]
        bias[hot.to(device)] += cfg.hot_bias
    return logits, bias, hot


def gen_router_weight(cfg: MoEConfig, seed: int, device="cpu"):
    """Router projection weight fp32 [E_g, H], N(0, 1/H)."""
    return torch.randn(cfg.num_experts, cfg.H, generator=_gen(device, seed, TID_ROUTER_W),
                       device=device, dtype=torch.float32) * (1.0 / cfg.H) ** 0.5


def gen_hidden(cfg: MoEConfig, seed: int, device="cpu"):
    """(hidden e4m3fn codes uint8 [T,H], hidden_scale fp32 [T,H/128])."""
    x = torch.randn(max(cfg.T, 1), cfg.H, generator=_gen(device, seed, TID_HIDDEN),
                    device=device, dtype=torch.float32)[: cfg.T]
    if cfg.T == 0:
        return (torch.empty(0, cfg.H, dtype=torch.uint8, device=device),
                torch.empty(0, cfg.H // 128, dtype=torch.float32, device=device))
    return quantize_blocks(x, 1, 128)


def gen_expert(cfg: MoEConfig, seed: int, e: int, device="cpu"):
    """Weights of local expert ``e``: (w13 [2I,H] u8, w13_scale [2I/128,H/128],
    w2 [H,I] u8, w2_scale [H/128,I/128]).  The sub-stream is keyed by the
    global expert id, so a slice regenerates the same bytes."""
    gid = cfg.local_expert_offset + e
    w13 = torch.randn(2 * cfg.I, cfg.H, generator=_gen(device, seed, TID_W13, gid),
                      device=device, dtype=torch.float32) * 0.02
    q13, s13 = quantize_blocks(w13, 128, 128)
    del w13
    w2 = torch.randn(cfg.H, cfg.I, generator=_gen(device, seed, TID_W2, gid),
                     device=device, dtype=torch.float32) * 0.02
    q2, s2 = quantize_blocks(w2, 128, 128)
    return q13, s13, q2, s2


def gen_weights(cfg: MoEConfig, seed: int, device="cpu"):
    """All resident experts stacked: (w13 [E_l,2I,H], w13_scale, w2 [E_l,H,I], w2_scale)."""
    El, H, I = cfg.num_local_experts, cfg.H, cfg.I
    w13 = torch.empty(El, 2 * I, H, dtype=torch.uint8, device=device)
    s13 = torch.empty(El, 2 * I // 128, H // 128, dtype=torch.float32, device=device)
    w2 = torch.empty(El, H, I, dtype=torch.uint8, device=device)
    s2 = torch.empty(El, H // 128, I // 128, dtype=torch.float32, device=device)
    for e in range(El):
        a, b, c, d = gen_expert(cfg, seed, e, device)
        w13[e].copy_(a)
        s13[e].copy_(b)
        w2[e].copy_(c)
        s2[e].copy_(d)
    return w13, s13, w2, s2


@dataclass
class MoEInputs:
    cfg: MoEConfig
    seed: int
    hidden: torch.Tensor
    hidden_scale: torch.Tensor
    logits: torch.Tensor
    bias: torch.Tensor
    w13: torch.Tensor
    w13_scale: torch.Tensor
    w2: torch.Tensor
    w2_scale: torch.Tensor
    hot: torch.Tensor


def generate(cfg: MoEConfig, seed: int = 0, device="cpu") -> MoEInputs:
    logits, bias, hot = gen_router(cfg, seed, device)
    hidden, hscale = gen_hidden(cfg, seed, device)
    w13, s13, w2, s2 = gen_weights(cfg, seed, device)
    return MoEInputs(cfg, seed, hidden, hscale, logits, bias, w13, s13, w2, s2, hot)


def host_arrays(inp: MoEInputs, experts=None) -> dict:
    """numpy host copies for the oracle; weights only for ``experts`` (all by default)."""
    El = inp.cfg.num_local_experts
    want = set(range(El)) if experts is None else set(int(e) for e in experts)

    def per_expert(t):
        return [t[e].cpu().numpy() if e in want else None for e in range(El)]

    return dict(hidden=inp.hidden.cpu().numpy(), hidden_scale=inp.hidden_scale.cpu().numpy(),
                logits=inp.logits.cpu().numpy(), bias=inp.bias.cpu().numpy(),
                w13=per_expert(inp.w13), w13_scale=per_expert(inp.w13_scale),
                w2=per_expert(inp.w2), w2_scale=per_expert(inp.w2_scale))


# ---------------------------------------------------------------------------
# DSA TopK Indexer (paper Section 3.1.3): FP8 queries with 64 heads of 128,
# a paged FP8 key cache (64 tokens per page) with per-token fp32 scales,
# per-head weights, sequence lengths and block tables.  The paper's contest
# workloads are not available; these seeded inputs stand in for them:
#   q        N(0,1) per (b, head) row, quantised to e4m3 with scale amax/448;
#            the row scale is folded into the head weight (the operator has
#            no query scale)                                            id 21
#   weights  N(0,1) * row scale / sqrt(64 * 128)                        id 22
#   K cache  N(0,1) per token, quantised to e4m3 with scale amax/448    id 23
#   block tables: each sequence's pages drawn without replacement from
#            the cache (a random permutation)                           id 24
# ---------------------------------------------------------------------------
TID_DSA_Q, TID_DSA_W, TID_DSA_K, TID_DSA_BT = 21, 22, 23, 24


@dataclass(frozen=True)
class IndexerConfig:
    name: str
    seq_lens: tuple
    num_heads: int = 64
    head_dim: int = 128
    page_size: int = 64
    topk: int = 2048

    @property
    def B(self) -> int:
        return len(self.seq_lens)

    @property
    def max_pages(self) -> int:
        return max(1, max((s + self.page_size - 1) // self.page_size for s in self.seq_lens))

    @property
    def num_pages(self) -> int:
        # every sequence's pages are distinct; a few spare pages
        return sum((s + self.page_size - 1) // self.page_size for s in self.seq_lens) + 8


INDEXER_CONFIGS: dict[str, IndexerConfig] = {
    # the paper's long-regime representative (appendix profile): bs 4,
    # max 36 pages; one sequence above TopK
    "dsa_paper_long": IndexerConfig("dsa_paper_long", (98, 91, 2241, 100)),
    # all sequences at or below TopK: the index-remap path only
    "dsa_short": IndexerConfig("dsa_short", (64, 1, 2048, 1984, 0, 700)),
    # long sequences, several far above TopK
    "dsa_long": IndexerConfig("dsa_long", (65536, 32768, 8192, 2049, 40000, 16384, 2048, 100)),
    # small parity cases around page and TopK edges (TopK 256 keeps the
    # oracle quick while the selection still has to cut)
    "dsa_small": IndexerConfig("dsa_small", (257, 256, 255, 1000, 63, 640, 2500), topk=256),
}


@dataclass
class IndexerInputs:
    cfg: IndexerConfig
    q: torch.Tensor            # [B, NH, D] uint8 (e4m3 codes)
    weights: torch.Tensor      # [B, NH] fp32
    k_cache: torch.Tensor      # [num_pages, PS, D] uint8
    k_scale: torch.Tensor      # [num_pages, PS] fp32
    block_table: torch.Tensor  # [B, max_pages] int32
    seq_lens: torch.Tensor     # [B] int32


def generate_indexer(cfg: IndexerConfig, seed: int = 0, device="cpu") -> IndexerInputs:
    B, NH, D, PS = cfg.B, cfg.num_heads, cfg.head_dim, cfg.page_size
    qf = torch.randn(B * NH, D, generator=_gen(device, seed, TID_DSA_Q), device=device)
    q, qs = quantize_blocks(qf, 1, D)
    w = torch.randn(B, NH, generator=_gen(device, seed, TID_DSA_W), device=device)
    w = (w * qs.reshape(B, NH) / (NH * D) ** 0.5).contiguous()
    kf = torch.randn(cfg.num_pages * PS, D, generator=_gen(device, seed, TID_DSA_K), device=device)
    kc, ksc = quantize_blocks(kf, 1, D)
    g = torch.Generator(device="cpu")
    g.manual_seed(substream_seed(seed, TID_DSA_BT))
    perm = torch.randperm(cfg.num_pages, generator=g).to(torch.int32)
    bt = torch.zeros(B, cfg.max_pages, dtype=torch.int32)
    at = 0
    for b, s in enumerate(cfg.seq_lens):
        n = (s + PS - 1) // PS
        bt[b, :n] = perm[at:at + n]
        at += n
    return IndexerInputs(cfg, q.reshape(B, NH, D).contiguous(), w,
                         kc.reshape(cfg.num_pages, PS, D).contiguous(),
                         ksc.reshape(cfg.num_pages, PS).contiguous(), bt.to(device),
                         torch.tensor(cfg.seq_lens, dtype=torch.int32, device=device))


# ---------------------------------------------------------------------------
# DSA Sparse Attention (paper Section 3.1.2): per query token, 16 heads of
# q_nope (512) and q_pe (64) against a paged KV cache of 512-wide Kc and
# 64-wide Kp entries, through a list of TopK sparse indices.  The contest
# workloads are not available; seeded inputs of the same shapes stand in:
#   q_nope, q_pe, Kc, Kp   N(0,1) rounded to bf16                 ids 31-34
#   indices  TopK distinct cache positions of the token's sequence (a
#            sequence of seq_len tokens over randomly permuted pages),
#            -1 past a short sequence's length                     id 35
#   sm_scale 1/sqrt(192) (DeepSeek-V3's 128 + 64 query head width)
# ---------------------------------------------------------------------------
TID_ATT_QN, TID_ATT_QP, TID_ATT_KC, TID_ATT_KP, TID_ATT_IDX = 31, 32, 33, 34, 35


@dataclass(frozen=True)
class AttentionConfig:
    name: str
    seq_lens: tuple            # one per query token
    num_heads: int = 16
    dc: int = 512
    dp: int = 64
    page_size: int = 64
    topk: int = 2048
    num_pages: int = 0         # 0: just enough for the sequences

    @property
    def T(self) -> int:
        return len(self.seq_lens)

    @property
    def pages(self) -> int:
        need = sum((s + self.page_size - 1) // self.page_size for s in self.seq_lens)
        return max(self.num_pages, need, 1)


ATTENTION_CONFIGS: dict[str, AttentionConfig] = {
    # the paper's long-regime representative: 8 tokens, 8462 cache pages
    "attn_long": AttentionConfig("attn_long", (60000,) * 8, num_pages=8462),
    # the single-token and two-token regimes of its dispatch table
    "attn_one": AttentionConfig("attn_one", (30000,)),
    "attn_two": AttentionConfig("attn_two", (9000, 5000)),
    # parity cases: short sequences (padding), TopK 256 and 2048
    "attn_small": AttentionConfig("attn_small", (100, 3000, 257, 1), topk=256),
    "attn_pad": AttentionConfig("attn_pad", (700, 2048, 1500, 4000)),
}


@dataclass
class AttentionInputs:
    cfg: AttentionConfig
    q_nope: torch.Tensor   # [T, H, 512] bf16
    q_pe: torch.Tensor     # [T, H, 64] bf16
    ckv: torch.Tensor      # [pages, PS, 512] bf16
    kpe: torch.Tensor      # [pages, PS, 64] bf16
    indices: torch.Tensor  # [T, topk] int32
    sm_scale: float


def generate_attention(cfg: AttentionConfig, seed: int = 0, device="cpu") -> AttentionInputs:
    T, H, PS = cfg.T, cfg.num_heads, cfg.page_size
    qn = torch.randn(T, H, cfg.dc, generator=_gen(device, seed, TID_ATT_QN), device=device).to(torch.bfloat16)
    qp = torch.randn(T, H, cfg.dp, generator=_gen(device, seed, TID_ATT_QP), device=device).to(torch.bfloat16)
    kc = torch.randn(cfg.pages, PS, cfg.dc, generator=_gen(device, seed, TID_ATT_KC), device=device).to(torch.bfloat16)
    kp = torch.randn(cfg.pages, PS, cfg.dp, generator=_gen(device, seed, TID_ATT_KP), device=device).to(torch.bfloat16)
    g = torch.Generator(device="cpu")
    g.manual_seed(substream_seed(seed, TID_ATT_IDX))
    perm = torch.randperm(cfg.pages, generator=g)
    idx = torch.full((T, cfg.topk), -1, dtype=torch.int32)
    for t, s in enumerate(cfg.seq_lens):
        n = (s + PS - 1) // PS
        pages = perm[torch.randint(0, cfg.pages - n + 1, (1,), generator=g).item():][:n]
        k = min(s, cfg.topk)
        pos = torch.randperm(s, generator=g)[:k]
        idx[t, :k] = (pages[pos // PS] * PS + pos % PS).to(torch.int32)
    return AttentionInputs(cfg, qn, qp, kc, kp, idx.to(device), 1.0 / 192 ** 0.5)
