"""Seeded synthetic inputs for one serving iteration's attention over a paged KV cache.

The batches mirror the iterations the paper schedules (Sections 3 and 4):
chunked-prefill segments with a cached prefix mixed with many single-token
decode requests, each request reading its keys and values through a page
table.  Shapes are those of Llama-3-8B and Llama-3-70B attention.

This module only draws numbers (request lengths, the physical page each
logical page lives in, Q/K/V values).  It holds none of the attention or
latency-model arithmetic, so both the GPU path and the CPU oracle can take
their inputs from it.

Cache layouts (one layer):
  k_cache  [num_phys_pages, h_kv, page_size, head_dim]   token-major pages
  v_cache  [num_phys_pages, h_kv, head_dim, page_size]   dim-major pages
Token t of request r lives in slot t % page_size of physical page
page_table[r, t // page_size].  Slots and pages that no request uses hold NaN.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

PAGE_SIZE = 16
KIND_PREFILL = 0
KIND_DECODE = 1


@dataclass(frozen=True)
class AttnShape:
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str  # "bf16" or "f32"
    page_size: int = PAGE_SIZE
    num_layers: int = 1

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4


LLAMA3_8B = AttnShape(32, 8, 128, "bf16")
LLAMA3_70B = AttnShape(64, 8, 128, "bf16")
TINY_F32 = AttnShape(4, 2, 64, "f32")


@dataclass
class Batch:
    """Host description of one mixed iteration: per-request lengths and page table."""

    shape: AttnShape
    kinds: np.ndarray  # int32 [R]
    q_lens: np.ndarray  # int32 [R]
    cached_lens: np.ndarray  # int32 [R]
    page_table: np.ndarray  # int32 [R, max_pages], -1 padded
    num_phys_pages: int
    name: str = ""
    meta: dict = field(default_factory=dict)

    @property
    def num_reqs(self) -> int:
        return int(self.kinds.shape[0])

    @property
    def q_starts(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.q_lens)[:-1]]).astype(np.int32)

    @property
    def kv_lens(self) -> np.ndarray:
        return (self.cached_lens + self.q_lens).astype(np.int64)

    @property
    def num_tokens(self) -> int:
        return int(self.q_lens.sum())

    @property
    def seq_meta(self) -> np.ndarray:
        """int32 [R, 4] rows of (kind, q_start, q_len, cached_len)."""
        return np.stack([self.kinds, self.q_starts, self.q_lens, self.cached_lens], axis=1).astype(np.int32)

    def pages_of(self, r: int) -> np.ndarray:
        n = -(-int(self.kv_lens[r]) // self.shape.page_size)
        return self.page_table[r, :n]

    def used_pages(self) -> np.ndarray:
        """Physical pages in logical order: request by request, page by page."""
        return np.concatenate([self.pages_of(r) for r in range(self.num_reqs)]).astype(np.int64)


def _assign_pages(n_pages_per_req, num_phys_pages, rng) -> np.ndarray:
    total = int(sum(n_pages_per_req))
    if total > num_phys_pages:
        raise ValueError(f"{total} pages needed, pool holds {num_phys_pages}")
    # A seeded injection of the used logical pages into the physical pool.
    chosen = rng.permutation(num_phys_pages)[:total] if num_phys_pages <= 1 << 24 else \
        rng.choice(num_phys_pages, size=total, replace=False)
    width = max(1, max(n_pages_per_req))
    table = np.full((len(n_pages_per_req), width), -1, dtype=np.int32)
    off = 0
    for r, n in enumerate(n_pages_per_req):
        table[r, :n] = chosen[off:off + n]
        off += n
    return table


def make_batch(shape: AttnShape, reqs, *, page_seed: int, num_phys_pages: int | None = None,
               pool_slack: float = 0.10, name: str = "", reserve_tokens: int = 0) -> Batch:
    """reqs: list of (kind, q_len, cached_len).  Pages are placed by a seeded permutation.
    reserve_tokens: decode requests also get pages for that many future tokens (the KV slots of
    look-ahead decode steps); those slots start out NaN."""
    kinds = np.array([k for k, _, _ in reqs], dtype=np.int32)
    q_lens = np.array([q for _, q, _ in reqs], dtype=np.int32)
    cached = np.array([c for _, _, c in reqs], dtype=np.int32)
    if np.any(q_lens < 1) or np.any(cached < 0):
        raise ValueError("q_len >= 1 and cached_len >= 0 required")
    ps = shape.page_size
    if reserve_tokens < 0:
        raise ValueError("reserve_tokens >= 0 required")
    n_pages = [-(-int(c + q + (reserve_tokens if k == KIND_DECODE else 0)) // ps)
               for k, q, c in zip(kinds, q_lens, cached)]
    if num_phys_pages is None:
        num_phys_pages = int(math.ceil(sum(n_pages) * (1.0 + pool_slack))) + 1
    rng = np.random.Generator(np.random.PCG64(page_seed))
    table = _assign_pages(n_pages, num_phys_pages, rng)
    return Batch(shape, kinds, q_lens, cached, table, int(num_phys_pages), name=name,
                 meta={"reserve_tokens": int(reserve_tokens)} if reserve_tokens else {})


# ----------------------------------------------------------------------------------------------
# The five workloads.  Host draws use PCG64 with seed = 1000 + workload number unless given.
# ----------------------------------------------------------------------------------------------

def tiny_mixed(seed: int = 1001, page_seed: int | None = None) -> Batch:
    """fp32, 4 q-heads / 2 kv-heads / head_dim 64, one 48-token chunk after a 16-token prefix
    plus decodes at context 17, 40 and 100, in a pool of 32 pages."""
    reqs = [(KIND_PREFILL, 48, 16), (KIND_DECODE, 1, 16), (KIND_DECODE, 1, 39), (KIND_DECODE, 1, 99)]
    return make_batch(TINY_F32, reqs, page_seed=seed if page_seed is None else page_seed,
                      num_phys_pages=32, name="tiny-mixed-f32")


def llama8b_mixed(seed: int = 1002, page_seed: int | None = None, num_decodes: int = 64,
                  prefill_len: int = 2048, reserve_tokens: int = 0) -> Batch:
    """Llama-3-8B shapes: a 2048-token prefill at prefix 0 plus 64 decodes, context U{512..4096}."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ctx = rng.integers(512, 4096, size=num_decodes, endpoint=True)
    reqs = [(KIND_PREFILL, prefill_len, 0)] + [(KIND_DECODE, 1, int(c) - 1) for c in ctx]
    return make_batch(LLAMA3_8B, reqs, page_seed=seed + 7 if page_seed is None else page_seed,
                      name="llama3-8b-mixed-2048p-64d", reserve_tokens=reserve_tokens)


def decode_heavy(seed: int = 1003, page_seed: int | None = None, num_decodes: int = 256,
                 pool_bytes: float = 70e9) -> Batch:
    """256 decodes with lognormal contexts (median 8192, sigma 0.8, cap 32768) plus a 512-token
    chunk after a 16384-token prefix; used pages scattered through a ~70 GB page pool."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ctx = np.minimum(32768, np.maximum(1, np.rint(rng.lognormal(math.log(8192.0), 0.8, size=num_decodes))))
    reqs = [(KIND_DECODE, 1, int(c) - 1) for c in ctx] + [(KIND_PREFILL, 512, 16384)]
    sh = LLAMA3_8B
    page_pair_bytes = 2 * sh.num_kv_heads * sh.page_size * sh.head_dim * sh.elem_bytes
    pool = int(pool_bytes // page_pair_bytes)
    return make_batch(sh, reqs, page_seed=seed + 7 if page_seed is None else page_seed,
                      num_phys_pages=pool, name="llama3-8b-decode-heavy-256d")


def prefill_heavy_70b(seed: int = 1004, page_seed: int | None = None, reserve_tokens: int = 0) -> Batch:
    """Llama-3-70B shapes: an 8192-token chunk after a 24576-token prefix plus 32 decodes at 2048.
    reserve_tokens: KV slots of that many future decode tokens per decode request (look-ahead)."""
    reqs = [(KIND_PREFILL, 8192, 24576)] + [(KIND_DECODE, 1, 2047)] * 32
    return make_batch(LLAMA3_70B, reqs, page_seed=seed + 7 if page_seed is None else page_seed,
                      name="llama3-70b-prefill-heavy", reserve_tokens=reserve_tokens)


WORKLOADS = {1: tiny_mixed, 2: llama8b_mixed, 3: decode_heavy, 4: prefill_heavy_70b}


# ----------------------------------------------------------------------------------------------
# Tensor values
# ----------------------------------------------------------------------------------------------

def value_scale(shape: AttnShape) -> float:
    """N(0,1) for the fp32 tiny case, N(0,1) * 0.1 for the bf16 model shapes."""
    return 1.0 if shape.dtype == "f32" else 0.1


def make_tensors(batch: Batch, seed: int, *, device="cpu", scale: float | None = None,
                 chunk_pages: int = 1 << 14):
    """Draw Q, then K, then V with a torch generator on `device`; returns (q, k_cache, v_cache).

    Values are drawn in logical order (request by request, page by page), so two batches that
    differ only in page placement hold the same logical sequences.  Slots past each request's
    length and pages no request uses are NaN.
    """
    import torch

    sh = batch.shape
    tdt = torch.bfloat16 if sh.dtype == "bf16" else torch.float32
    scale = value_scale(sh) if scale is None else scale
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(int(seed))
    ps, hk, d = sh.page_size, sh.num_kv_heads, sh.head_dim

    q = (torch.randn(batch.num_tokens, sh.num_q_heads, d, generator=gen, device=dev) * scale).to(tdt)
    k_cache = torch.full((batch.num_phys_pages, hk, ps, d), float("nan"), dtype=tdt, device=dev)
    v_cache = torch.full((batch.num_phys_pages, hk, d, ps), float("nan"), dtype=tdt, device=dev)
    used = torch.as_tensor(batch.used_pages(), device=dev)
    # Tail slot mask per used page (logical order): slots >= valid count become NaN.
    valid = []
    for r in range(batch.num_reqs):
        L = int(batch.kv_lens[r])
        n = -(-L // ps)
        v = np.full(n, ps, dtype=np.int64)
        v[-1] = L - (n - 1) * ps
        valid.append(v)
    valid = torch.as_tensor(np.concatenate(valid), device=dev)
    slot = torch.arange(ps, device=dev)
    for which, cache in (("k", k_cache), ("v", v_cache)):
        for lo in range(0, used.numel(), chunk_pages):
            hi = min(used.numel(), lo + chunk_pages)
            vals = (torch.randn(hi - lo, hk, ps, d, generator=gen, device=dev) * scale).to(tdt)
            dead = (slot[None, :] >= valid[lo:hi, None])  # [n, ps]
            vals = vals.masked_fill(dead[:, None, :, None], float("nan"))
            if which == "v":
                vals = vals.transpose(2, 3).contiguous()
            cache[used[lo:hi]] = vals
    return q, k_cache, v_cache


def make_lookahead_tensors(batch: Batch, k: int, seed: int, *, device="cpu", scale: float | None = None):
    """Inputs of look-ahead decode steps 1 .. k - 1 for one layer: lists (one tensor per step) of
    queries [R_d, h_q, d] and new key / value rows [R_d, h_kv, d], decode requests in batch order,
    drawn in that order (per step: q, then k, then v) with a torch generator on `device`."""
    import torch

    sh = batch.shape
    tdt = torch.bfloat16 if sh.dtype == "bf16" else torch.float32
    scale = value_scale(sh) if scale is None else scale
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(int(seed))
    n_dec = int((batch.kinds == KIND_DECODE).sum())
    qa, ka, va = [], [], []
    for _ in range(k - 1):
        qa.append((torch.randn(n_dec, sh.num_q_heads, sh.head_dim, generator=gen, device=dev) * scale).to(tdt))
        ka.append((torch.randn(n_dec, sh.num_kv_heads, sh.head_dim, generator=gen, device=dev) * scale).to(tdt))
        va.append((torch.randn(n_dec, sh.num_kv_heads, sh.head_dim, generator=gen, device=dev) * scale).to(tdt))
    return qa, ka, va


# ----------------------------------------------------------------------------------------------
# Serving trace: seeded arrivals and lengths, decode-first token-budget batch formation
# ----------------------------------------------------------------------------------------------

def lognormal_mean_params(mean: float, sigma: float):
    """(mu, sigma) of a lognormal whose mean (not median) is `mean`."""
    return math.log(mean) - sigma * sigma / 2.0, sigma


@dataclass
class _Live:
    rid: int
    prompt: int
    output: int
    prefilled: int = 0
    generated: int = 0


def trace_requests(seed: int = 1005, *, rate: float = 4.0, prompt_mean: float = 4096, prompt_sigma: float = 1.0,
                   output_mean: float = 256, output_sigma: float = 0.7, cap: int = 32768, n_req: int = 200000):
    """The request stream of the serving trace: Poisson arrival times (s), lognormal prompt and output
    lengths (means as given, clipped to [1, cap]), drawn in that order from PCG64(seed)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    pmu, psg = lognormal_mean_params(prompt_mean, prompt_sigma)
    omu, osg = lognormal_mean_params(output_mean, output_sigma)
    gaps = rng.exponential(1.0 / rate, size=n_req)
    arrivals = np.cumsum(gaps)
    prompts = np.clip(np.rint(rng.lognormal(pmu, psg, size=n_req)), 1, cap).astype(np.int64)
    outputs = np.clip(np.rint(rng.lognormal(omu, osg, size=n_req)), 1, cap).astype(np.int64)
    return arrivals, prompts, outputs


def serving_trace(num_iters: int = 200, seed: int = 1005, *, rate: float = 4.0, prompt_mean: float = 4096,
                  prompt_sigma: float = 1.0, output_mean: float = 256, output_sigma: float = 0.7,
                  cap: int = 32768, token_budget: int = 8192, warmup_iters: int = 200,
                  iter_seconds=lambda reqs: 0.05):
    """Batches of a synthetic serving run: Poisson arrivals, lognormal prompt/output lengths and
    a chunked-prefill scheduler that admits every running decode first (one token each) and then
    fills the rest of the token budget with prefill tokens, chunking the last prompt.

    Returns a list of request lists [(kind, q_len, cached_len), ...], one per recorded iteration,
    after `warmup_iters` unrecorded iterations.  `iter_seconds(reqs)` advances the clock.
    """
    arrivals, prompts, outputs = trace_requests(seed, rate=rate, prompt_mean=prompt_mean, prompt_sigma=prompt_sigma,
                                                output_mean=output_mean, output_sigma=output_sigma, cap=cap)
    n_req = len(arrivals)
    clock = 0.0
    nxt = 0
    waiting: list[_Live] = []
    running: list[_Live] = []
    out = []
    for it in range(warmup_iters + num_iters):
        while nxt < n_req and arrivals[nxt] <= clock:
            waiting.append(_Live(nxt, int(prompts[nxt]), int(outputs[nxt])))
            nxt += 1
        if not waiting and not running and nxt < n_req:
            clock = float(arrivals[nxt])
            continue
        reqs = []
        budget = token_budget
        decodes = [r for r in running if r.prefilled >= r.prompt]
        for r in decodes[:budget]:
            ctx = r.prompt + r.generated
            reqs.append((KIND_DECODE, 1, ctx))
            budget -= 1
        chunks = []
        partial = [r for r in running if r.prefilled < r.prompt]
        for r in partial + waiting:
            if budget <= 0:
                break
            take = min(budget, r.prompt - r.prefilled)
            reqs.append((KIND_PREFILL, take, r.prefilled))
            chunks.append((r, take))
            budget -= take
        for r, take in chunks:
            if r in waiting:
                waiting.remove(r)
                running.append(r)
            r.prefilled += take
        for r in decodes[:token_budget]:
            r.generated += 1
        running = [r for r in running if r.generated < r.output]
        if it >= warmup_iters and reqs:
            out.append(reqs)
        clock += float(iter_seconds(reqs))
        if len(out) >= num_iters:
            break
    return out


def block_weights(sh: AttnShape, ffn_dim: int, layers: int, gen):
    """Per-layer bf16 weight dicts drawn from the torch generator `gen` (on its device), per layer
    in the order attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down: norm weights 1 + 0.1 N(0,1),
    a [d_in, d_out] matrix N(0,1) / sqrt(d_in)."""
    import torch

    dev = gen.device
    d = sh.num_q_heads * sh.head_dim
    d_qkv = (sh.num_q_heads + 2 * sh.num_kv_heads) * sh.head_dim
    m = int(ffn_dim)

    def mat(d_in, d_out):
        return (torch.randn(d_in, d_out, generator=gen, device=dev) / math.sqrt(d_in)).to(torch.bfloat16)

    def norm_w(n):
        return (1.0 + 0.1 * torch.randn(n, generator=gen, device=dev)).to(torch.bfloat16)

    return [{"attn_norm": norm_w(d), "w_qkv": mat(d, d_qkv), "w_o": mat(d, d), "ffn_norm": norm_w(d),
             "w_gate_up": mat(d, 2 * m), "w_down": mat(m, d)} for _ in range(layers)]


def make_block_tensors(batch: Batch, ffn_dim: int, layers: int, seed: int, *, device="cpu"):
    """Inputs of an L-block forward (bf16): the residual stream x [T, h_q d], per-layer weight
    dicts and per-layer (k_cache, v_cache).  Drawn with a torch generator on `device`, in this
    order: x, then per layer attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down; the caches come
    from make_tensors with seed + 1 + l.  Norm weights are 1 + 0.1 N(0,1); a [d_in, d_out] matrix
    is N(0,1) / sqrt(d_in); x is N(0,1).  The new tokens' cache slots hold values the forward
    overwrites."""
    import torch

    sh = batch.shape
    if sh.dtype != "bf16":
        raise ValueError("the block inputs are bf16")
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(int(seed))
    d = sh.num_q_heads * sh.head_dim
    m = int(ffn_dim)
    x = torch.randn(batch.num_tokens, d, generator=gen, device=dev).to(torch.bfloat16)
    weights = block_weights(sh, m, layers, gen)
    caches = []
    for l in range(layers):
        _, kc, vc = make_tensors(batch, seed + 1 + l, device=device)
        caches.append((kc, vc))
    return x, weights, caches


def make_block_ahead(batch: Batch, k: int, seed: int, *, device="cpu"):
    """Residual rows of look-ahead decode steps 1 .. k - 1 for an L-block forward: k - 1 bf16
    tensors [R_d, h_q d] (decode requests in batch order), N(0,1), drawn in step order with a
    torch generator on `device`."""
    import torch

    sh = batch.shape
    n_dec = int((batch.kinds == KIND_DECODE).sum())
    gen = torch.Generator(device=torch.device(device))
    gen.manual_seed(int(seed))
    d = sh.num_q_heads * sh.head_dim
    return [torch.randn(n_dec, d, generator=gen, device=torch.device(device)).to(torch.bfloat16)
            for _ in range(k - 1)]
