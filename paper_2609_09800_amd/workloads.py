"""Seeded synthetic request streams and GEMV operands.

This module only draws inputs: addresses, issue times and bf16 operands.  It
holds none of the service model's arithmetic (no classification, no mapping,
no queueing) and is shared, as a pure input source, by the HIP path's tests,
the reference model's tests and the benchmark.

The paper's workloads (Qwen3-30B-A3B decode under vLLM, a captured routing
trace; Section "Evaluation", EQ1 and EQ3) are not available, so every stream
here is a seeded stand-in with the shape the paper describes: 48 MoE layers of
128 experts with top-8 routing, expert weights streamed as 16 KiB page reads,
and a shared read-mostly KV prefix (a system prompt) that HBF suits
(Section "Background", first observation).

All draws use ``numpy.random.Generator(PCG64(seed))`` in a fixed order, so the
same seed yields bit-identical arrays on every machine with this numpy.
"""
from dataclasses import dataclass, field

import numpy as np

KIB = 1024
GIB = 1 << 30
TIB = 1 << 40
PAGE = 16 * KIB
RANGE_BASE = 1 << 40

# Qwen3-30B-A3B-shaped MoE (48 layers, 128 experts, top-8, hidden 2048,
# expert FFN 768): one expert is three bf16 matrices, 2048x768, 2048x768 and
# 768x2048.  48*128 such experts are the paper's 54.000 GiB expert set
# (Section "Evaluation", EQ3).
MOE_LAYERS = 48
MOE_EXPERTS = 128
MOE_TOPK = 8
MOE_HIDDEN = 2048
MOE_FFN = 768
EXPERT_BYTES = 3 * MOE_HIDDEN * MOE_FFN * 2
PAGES_PER_EXPERT = EXPERT_BYTES // PAGE  # 576
ZIPF_S = 1.1

# Shared KV prefix: 4096-token system prompt, 48 layers x 4 KV heads x 128
# dim, bf16, K and V.
KV_TOKENS = 4096
KV_HEADS = 4
KV_DIM = 128
KV_BYTES = KV_TOKENS * MOE_LAYERS * KV_HEADS * KV_DIM * 2 * 2
KV_PAGES = KV_BYTES // PAGE  # 24576


def geometry(channels, dies, planes, t_read_ns=3000, bw=8_000_000_000, page=PAGE, flags=0):
    return dict(channels=channels, dies_per_channel=dies, planes_per_die=planes, page_bytes=page,
                t_read_ns=t_read_ns, channel_bytes_per_s=bw, flags=flags)


@dataclass
class Workload:
    name: str
    params: dict
    ranges: list
    addr: np.ndarray
    issue: np.ndarray
    meta: dict = field(default_factory=dict)

    @property
    def n(self):
        return int(self.addr.size)


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def poisson_issue(rng, n, mean_gap):
    """Open-loop arrivals: gaps floor(Exponential(mean)) ns, cumulated (ties allowed)."""
    if n == 0:
        return np.zeros(0, dtype=np.int64)
    gaps = np.floor(rng.exponential(mean_gap, n)).astype(np.int64)
    return np.cumsum(gaps, dtype=np.int64)


def config1(seed=0):
    """4,096 page reads, 8ch x 4 die x 1 plane, tR 3000 ns, 4 GB/s per channel.

    90 % uniform pages of a 1 GiB range at 2^40; the other 10 % are uniform
    pages of the 1 GiB windows just below (half) and just above (half) it.
    Poisson arrivals with mean gap 200 ns.
    """
    rng = _rng(seed)
    n = 4096
    rbytes = GIB
    pages = rbytes // PAGE
    u = rng.random(n)
    pg = rng.integers(0, pages, n, dtype=np.int64).astype(np.uint64)
    addr = np.uint64(RANGE_BASE) + pg * np.uint64(PAGE)
    above = (u >= 0.9) & (u < 0.95)
    below = u >= 0.95
    addr[above] += np.uint64(rbytes)
    addr[below] -= np.uint64(rbytes)
    issue = poisson_issue(rng, n, 200.0)
    return Workload("config1-tiny-stream", geometry(8, 4, 1, bw=4_000_000_000), [(RANGE_BASE, rbytes)],
                    addr, issue)


def config2(seed=0, n=1 << 20):
    """1,048,576 reads, 16ch x 8 die x 4 plane, tR 3000 ns, 8 GB/s, 64 GiB range.

    Segments: with p = 32/33 one uniform page, otherwise a sequential run from
    a uniform page of length Geometric(1/32) clamped to [1, 256], wrapping
    modulo the range.  About half the requests come from each.  Poisson
    arrivals with mean gap 20 ns.
    """
    rng = _rng(seed)
    rbytes = 64 * GIB
    pages = rbytes // PAGE
    m = n  # enough segments: every segment has length >= 1
    single = rng.random(m) < 32.0 / 33.0
    runlen = np.clip(rng.geometric(1.0 / 32.0, m), 1, 256)
    L = np.where(single, 1, runlen).astype(np.int64)
    start = rng.integers(0, pages, m, dtype=np.int64)
    cum = np.cumsum(L)
    k = int(np.searchsorted(cum, n)) + 1
    L = L[:k]
    start = start[:k]
    seg = np.repeat(np.arange(k), L)[:n]
    off = np.arange(n, dtype=np.int64) - np.repeat(cum[:k] - L, L)[:n]
    pg = (start[seg] + off) % pages
    addr = np.uint64(RANGE_BASE) + pg.astype(np.uint64) * np.uint64(PAGE)
    issue = poisson_issue(rng, n, 20.0)
    return Workload("config2-1M-uniform-runs", geometry(16, 8, 4), [(RANGE_BASE, rbytes)], addr, issue,
                    meta=dict(single_share=float(np.mean(L[single[:k]] == 1)) if k else 0.0))


class MoeRouter:
    """Zipf(s = 1.1) expert popularity with a fixed per-layer permutation.

    Each of ``tokens`` tokens picks ``topk`` distinct experts, weighted,
    without replacement.  Drawn with the Gumbel-top-k construction, which
    samples exactly the sequential weighted-without-replacement distribution.
    """

    def __init__(self, rng, layers=MOE_LAYERS, experts=MOE_EXPERTS, topk=MOE_TOPK, s=ZIPF_S):
        self.rng = rng
        self.layers, self.experts, self.topk = layers, experts, topk
        w_rank = np.arange(1, experts + 1, dtype=np.float64) ** (-s)
        self.logw = np.empty((layers, experts))
        for l in range(layers):
            perm = rng.permutation(experts)  # perm[r] = expert at popularity rank r
            self.logw[l, perm] = np.log(w_rank)

    def route(self, tokens):
        """Per layer: (tokens x topk) expert ids for one decode step."""
        g = self.rng.gumbel(size=(self.layers, tokens, self.experts))
        keys = self.logw[:, None, :] + g
        return np.argpartition(-keys, self.topk - 1, axis=2)[:, :, :self.topk]

    def active(self, tokens):
        """Per layer: the sorted union of experts any token routed to."""
        ch = self.route(tokens)
        return [np.unique(ch[l]) for l in range(self.layers)]


def moe_step_pages(active_per_layer):
    """Page indices of one decode step: layer order, experts ascending, pages in order.

    Expert (l, e) occupies pages [(l*128 + e)*576, +576) of the range.
    """
    out, lay = [], []
    for l, act in enumerate(active_per_layer):
        first = (l * MOE_EXPERTS + act.astype(np.int64)) * PAGES_PER_EXPERT
        pg = (first[:, None] + np.arange(PAGES_PER_EXPERT, dtype=np.int64)[None, :]).ravel()
        out.append(pg)
        lay.append(np.full(pg.size, l, dtype=np.int64))
    return np.concatenate(out), np.concatenate(lay)


def config3(seed=0, steps=16, tokens=64):
    """MoE decode weight streaming, 16 steps of a 64-token batch.

    Every active expert's 576 pages are issued at (s*48 + l) * 2000 ns: 2 us of
    compute spacing per layer, open loop.  16ch x 8 die x 4 plane, tR 3000 ns,
    8 GB/s, over the 54 GiB expert range.
    """
    rng = _rng(seed)
    router = MoeRouter(rng)
    pages, issue, per_layer = [], [], []
    for s in range(steps):
        act = router.active(tokens)
        per_layer.append([a.size for a in act])
        pg, lay = moe_step_pages(act)
        pages.append(pg)
        issue.append((s * MOE_LAYERS + lay) * 2000)
    pg = np.concatenate(pages)
    addr = np.uint64(RANGE_BASE) + pg.astype(np.uint64) * np.uint64(PAGE)
    rbytes = MOE_LAYERS * MOE_EXPERTS * EXPERT_BYTES
    return Workload("config3-moe-decode", geometry(16, 8, 4), [(RANGE_BASE, rbytes)], addr,
                    np.concatenate(issue).astype(np.int64),
                    meta=dict(active_per_layer=np.array(per_layer)))


def config3_layers(seed=0, steps=2, tokens=64):
    """The config-3 decode as a closed loop: the same pages, grouped per
    (step, layer) in program order, for issue times that follow the modeled
    completions.  Returns (workload with issue times zero, layer_start[L+1])."""
    rng = _rng(seed)
    router = MoeRouter(rng)
    pages, sizes = [], []
    for s in range(steps):
        act = router.active(tokens)
        pg, lay = moe_step_pages(act)
        pages.append(pg)
        sizes.extend(np.bincount(lay, minlength=MOE_LAYERS).tolist())
    pg = np.concatenate(pages)
    addr = np.uint64(RANGE_BASE) + pg.astype(np.uint64) * np.uint64(PAGE)
    rbytes = MOE_LAYERS * MOE_EXPERTS * EXPERT_BYTES
    ls = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    w = Workload("config3-moe-decode-closed-loop", geometry(16, 8, 4), [(RANGE_BASE, rbytes)], addr,
                 np.zeros(addr.size, dtype=np.int64))
    return w, ls


def dedup_demand(seed=0, batches=(1, 8, 16), steps=16):
    """Mean deduplicated active experts per layer at several batch sizes
    (the quantity of the paper's MoE-demand figure, EQ3)."""
    out = {}
    for b in batches:
        router = MoeRouter(_rng(seed))
        tot = 0
        for _ in range(steps):
            tot += sum(a.size for a in router.active(b))
        out[b] = tot / (steps * MOE_LAYERS)
    return out


def bf16_bits(x):
    """Round float32 values to bfloat16 (round to nearest even); return the bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def config4_operands(seed=0, batch=1, experts=8, K=MOE_HIDDEN, N=MOE_FFN):
    """bf16 weights W[e][n][k] ~ N(0,1)/sqrt(K) and activations X[e][b][k] ~ N(0,1)."""
    rng = _rng(seed)
    W = bf16_bits(rng.standard_normal((experts, N, K), dtype=np.float32) / np.float32(np.sqrt(K)))
    X = bf16_bits(rng.standard_normal((experts, batch, K), dtype=np.float32))
    return W, X


def config4_experts(seed=0):
    """The 8 experts most chosen at step 0, layer 0 of the config-3 router
    (the experts whose weights the instrumented GEMV stands in for)."""
    router = MoeRouter(_rng(seed))
    ch = router.route(64)[0].ravel()
    cnt = np.bincount(ch, minlength=MOE_EXPERTS)
    return np.argsort(-cnt, kind="stable")[:8]


def config4_pages(w_base, n_pages=1536):
    """One page read per 16 KiB weight page, all issued at time 0, on a reset model."""
    addr = np.uint64(w_base) + np.arange(n_pages, dtype=np.uint64) * np.uint64(PAGE)
    return addr, np.zeros(n_pages, dtype=np.int64)


def config5(seed=0, n=1 << 28):
    """Large mixed stream: 2^28 reads, 32ch x 16 die x 4 plane, 1 TiB range.

    80 % are MoE weight pages generated as in config 3 (continued over as many
    decode steps as needed), 20 % are reads of the shared KV prefix at offset
    64 GiB, sweeping its pages layer 0 -> 47 in order and repeating.
    Poisson arrivals with mean gap 2 ns.
    """
    rng = _rng(seed)
    is_kv = rng.random(n) < 0.2
    n_kv = int(np.count_nonzero(is_kv))
    n_moe = n - n_kv
    router = MoeRouter(rng)
    chunks, got = [], 0
    while got < n_moe:
        pg, _ = moe_step_pages(router.active(64))
        chunks.append(pg)
        got += pg.size
    moe = np.concatenate(chunks)[:n_moe]
    del chunks
    steps = None
    pages = np.empty(n, dtype=np.int64)
    pages[~is_kv] = moe
    del moe
    kv_first = 64 * GIB // PAGE
    pages[is_kv] = kv_first + (np.arange(n_kv, dtype=np.int64) % KV_PAGES)
    del is_kv
    addr = pages.view(np.uint64)
    addr *= np.uint64(PAGE)
    addr += np.uint64(RANGE_BASE)
    issue = poisson_issue(rng, n, 2.0)
    return Workload("config5-large-mixed", geometry(32, 16, 4), [(RANGE_BASE, TIB)], addr, issue,
                    meta=dict(n_kv=n_kv, steps=steps))


def capacity_stream(seed=0, steps=1, tokens=64):
    """Config 3's decode as a capacity-mode stream (Section D5): the expert
    set (48 x 128 experts x 576 pages) is one capacity range and every
    access is a page number within it, in program order.  Returns (pages
    int64, range_pages)."""
    rng = _rng(seed)
    router = MoeRouter(rng)
    out = []
    for _ in range(steps):
        pg, _lay = moe_step_pages(router.active(tokens))
        out.append(pg)
    return np.concatenate(out).astype(np.int64), MOE_LAYERS * MOE_EXPERTS * PAGES_PER_EXPERT


def config5_refresh_blocks(seed=0):
    """A refresh plan for the large mixed stream's device (32 ch x 16 die x
    4 plane), Section D4: epoch 0 makes one block of every plane eligible
    (zone = plane mod 2), epoch 1 one more plane-0 block of a random half of
    the dies; 32 pages per block, block indices uniform in [0, 1024).  The
    paper gives no program time; tPROG = 30,000 ns (10 tR) is assumed.
    Returns (blocks, pages_per_block, t_prog_ns)."""
    rng = _rng(seed + 5)
    blocks = []
    for ch in range(32):
        for die in range(16):
            for plane in range(4):
                blocks.append((0, plane % 2, ch, die, plane, int(rng.integers(0, 1024))))
    again = rng.random((32, 16)) < 0.5
    for ch in range(32):
        for die in range(16):
            if again[ch, die]:
                blocks.append((1, 0, ch, die, 0, int(rng.integers(0, 1024))))
    return blocks, 32, 30_000


def random_stream(seed, n, params, range_pages, mean_gap, out_frac=0.0, run_frac=0.0,
                  hot_dies=None, base=RANGE_BASE, burst=None):
    """Generic seeded stream for the parity suite.

    ``range_pages`` pages at ``base``; ``out_frac`` of requests fall just
    outside the range; ``run_frac`` of requests continue a sequential run from
    the previous one; ``hot_dies`` (if given) restricts page draws to
    pages = k * stride + offset so few resources see the traffic;
    ``burst`` = (count, at) places ``count`` requests at issue time ``at``.
    """
    rng = _rng(seed)
    page = params["page_bytes"]
    pg = rng.integers(0, range_pages, n, dtype=np.int64)
    if run_frac > 0 and n > 1:
        cont = rng.random(n) < run_frac
        cont[0] = False
        # a run continues the previous page: propagate from run starts
        idx = np.where(cont, 0, np.arange(n))
        np.maximum.accumulate(idx, out=idx)
        pg = (pg[idx] + (np.arange(n) - idx)) % range_pages
    if hot_dies is not None:
        stride, k = hot_dies
        pg = (pg // stride) * stride + (pg % k)
        pg %= range_pages
    addr = np.uint64(base) + pg.astype(np.uint64) * np.uint64(page)
    if out_frac > 0:
        o = rng.random(n) < out_frac
        side = rng.random(n) < 0.5
        span = np.uint64(range_pages * page)
        addr[o & side] += span
        addr[o & ~side] -= np.minimum(addr[o & ~side], span)
    issue = poisson_issue(rng, n, mean_gap)
    if burst is not None:
        cnt, at = burst
        issue = np.sort(np.concatenate([issue[:n - cnt], np.full(cnt, at, dtype=np.int64)]))
    return Workload(f"random-{seed}", dict(params), [(base, range_pages * page)], addr, issue)


ALL_CONFIGS = {1: config1, 2: config2, 3: config3, 5: config5}


# An illustrative calibrated vmem curve for the vmem timing source (T(L) in
# ns at 1, 4, 16, 64, 256 and 512 pages).  Only the first value is the
# paper's (the single-page cost it prints); the others are inputs of this
# project's workloads, chosen to cheapen the pages of a sequential burst
# until 64 pages and rise faster beyond, not values from the paper.
VMEM_KNOTS = (11_133, 14_500, 26_000, 80_000, 300_000, 640_000)
