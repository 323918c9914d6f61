"""Attention-aware roofline latency model and the CU-split choice, in plain Python doubles.

TEST INFRASTRUCTURE ONLY: the checker for the library's host-side predictor and optimiser.
Only the tests, the smoke check and the benchmark's CPU-baseline leg may use it.  It shares
no code with the C++ implementation.

Paper, Section 4.1 ("Sequence-Level Operators", "Overall Estimation"):
  F_attn/req(q, c) = 4 h_q q (q + c) d_h + 2 h_q q (q + c)           FLOPs
  B_attn/req(q, c) = 2 h_q q d_h b + 2 h_kv (q + c) d_h b               bytes
  t_attn = sum over requests of max(F / Pi, B / B_HBM)
  t_total = L * t_block, restricted here to the attention term of each of the L layers.
Paper, Section 4.2 and Algorithm 1:
  aggregated if t_mixed(S) <= tau; otherwise for each decode share S_d with t_d(S_d) <= tau,
  S_p = S - S_d, k in (floor(t_p / t_d), floor(t_p / t_d) + 1) and
  rho = (k T_decode + T_prefill) / max(k t_d, t_p); keep the first strictly larger rho.

Full-model estimate (Section 4.1, "Token-Level Operators", "Overall Estimation"):
  F_lin = 2 n d_i d_o,  B_lin = n d_i b + d_i d_o b + n d_o b  for n tokens through a d_i x d_o weight;
  QKV and output projections d -> d, gate-up d -> m, down m -> d (as the paper states them);
  t_tok = max(F_tok / Pi, B_tok / B_HBM) per operator, summed; t_block = t_tok + t_attn (one GPU:
  no all-reduce); t_total = L t_block + t_cls with t_cls a linear operator d -> vocab_size.
  Readings: RMSNorm F = 4 n d, B = 2 n d b + d b; SwiGLU activation F = 5 n m, B = 3 n m b;
  residual add F = n d, B = 3 n d b; the classifier runs on one row per request; options give the
  true GQA QKV width (h_q + 2 h_kv) d_h and a fused gate-up of width 2 m.

Extension (zero by default, which leaves the paper's model): a fixed latency per layer of each
partition kind on S CUs -- kernel launches and the decode kernel's tail, which no roofline
term sees -- added once per layer when the requests priced hold that kind.

Readings where the paper is silent (each also listed in the design notes):
  * The paper steps S_d by one TPC.  On MI355X the step is 32 CUs, S_d = 32, 64, ..., S - 32: a
    CU-mask bit b selects a CU on XCD b mod 8 and shader engine (b / 8) mod 4, the dispatcher
    deals a kernel's workgroups evenly to the shader engines of each XCD, and only multiples of
    32 give every shader engine of every XCD the same number of CUs (measured: a decode share of
    168 CUs runs 32% slower than one of 160).  The tables stay indexed by multiples of 8.
  * k = 0 is dropped: decode must make progress; k may be capped by the look-ahead depth.
  * No feasible S_d: fall back to aggregated execution and flag SLO_INFEASIBLE.
  * T_decode = number of decode requests; T_prefill = sum of the prefill requests' q.
  * b = 2 bytes for bf16, 4 for fp32; times in seconds here, microseconds at the C boundary.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

TOTAL_CUS = 256
CU_STEP = 8       # table index step: any multiple of 8 is a valid share
SPLIT_STEP = 32   # the S_d grid Algorithm 1 searches
NOMINAL_BF16_FLOPS = 2.5e15      # dense bf16 MFMA peak, FLOP/s
NOMINAL_HBM_BYTES = 8.0e12       # HBM3E bandwidth, B/s

AGG, SPLIT = 0, 1
SLO_INFEASIBLE = 1


def attn_flops(q: int, c: int, h_q: int, d_h: int) -> float:
    """F_attn/req: the QK^T and PV products over the q x (q + c) score block, plus softmax and scaling."""
    return 4.0 * h_q * q * (q + c) * d_h + 2.0 * h_q * q * (q + c)


def attn_bytes(q: int, c: int, h_q: int, h_kv: int, d_h: int, b: int) -> float:
    """B_attn/req: query read and output write, plus the key and value reads of all q + c tokens."""
    return 2.0 * h_q * q * d_h * b + 2.0 * h_kv * (q + c) * d_h * b


@dataclass
class Tables:
    """Achievable compute (FLOP/s) and HBM bandwidth (B/s) as functions of the CU count, and the
    fixed seconds per layer of each partition kind (absent: zero, the paper's model)."""
    flops: dict
    bw: dict
    launch_prefill: dict = None
    launch_decode: dict = None

    def pi(self, s: int) -> float:
        return self.flops[s]

    def b(self, s: int) -> float:
        return self.bw[s]

    def launch(self, kinds, s: int) -> float:
        """Fixed seconds per layer for a set of requests holding the given kinds (0 prefill, 1 decode)."""
        t = 0.0
        if 0 in kinds and self.launch_prefill:
            t += self.launch_prefill[s]
        if 1 in kinds and self.launch_decode:
            t += self.launch_decode[s]
        return t


def nominal_tables() -> Tables:
    cus = range(CU_STEP, TOTAL_CUS + 1, CU_STEP)
    return Tables({s: NOMINAL_BF16_FLOPS * s / TOTAL_CUS for s in cus},
                  {s: NOMINAL_HBM_BYTES * s / TOTAL_CUS for s in cus})


def t_attn(reqs, s: int, tables: Tables, h_q: int, h_kv: int, d_h: int, b: int) -> float:
    """Seconds for one layer's attention of the requests [(q, c), ...] on s CUs."""
    pi, bw = tables.pi(s), tables.b(s)
    return sum(max(attn_flops(q, c, h_q, d_h) / pi, attn_bytes(q, c, h_q, h_kv, d_h, b) / bw)
               for q, c in reqs)


def f_roofline(reqs, s, tables, *, h_q, h_kv, d_h, b, layers, kinds=()) -> float:
    """Seconds for the attention of all `layers` layers (t_total = L t_block, attention only);
    `kinds`: the request kinds present, whose fixed per-layer latency is added."""
    return layers * (t_attn(reqs, s, tables, h_q, h_kv, d_h, b) + tables.launch(kinds, s))


def kinds_of(batch):
    return {k for k, _, _ in batch}


def split_requests(batch):
    """batch: [(kind, q, c), ...] with kind 0 = prefill, 1 = decode."""
    pre = [(q, c) for k, q, c in batch if k == 0]
    dec = [(q, c) for k, q, c in batch if k == 1]
    return pre, dec


def predict(batch, mode, s_p, s_d, k, tables, *, h_q, h_kv, d_h, b, layers, total=TOTAL_CUS) -> float:
    """Predicted iteration latency in seconds: aggregated on all CUs, or max(k t_d(S_d), t_p(S_p))."""
    kw = dict(h_q=h_q, h_kv=h_kv, d_h=d_h, b=b, layers=layers)
    if mode == AGG:
        return f_roofline([(q, c) for _, q, c in batch], total, tables, kinds=kinds_of(batch), **kw)
    pre, dec = split_requests(batch)
    t_d = f_roofline(dec, s_d, tables, kinds={1}, **kw) if dec else 0.0
    t_p = f_roofline(pre, s_p, tables, kinds={0}, **kw) if pre else 0.0
    return max(k * t_d, t_p)


def choose(batch, tau, tables, *, h_q, h_kv, d_h, b, layers, total=TOTAL_CUS, step=SPLIT_STEP, kmax=None):
    """Algorithm 1.  Returns dict(mode, s_p, s_d, k, rho, t, flags).  kmax caps k at the number of
    decode steps the engine can launch ahead (Section 4.3): the two candidates are clamped to it;
    None leaves them as the paper states."""
    kw = dict(h_q=h_q, h_kv=h_kv, d_h=d_h, b=b, layers=layers)
    mixed = [(q, c) for _, q, c in batch]
    t_mixed = f_roofline(mixed, total, tables, kinds=kinds_of(batch), **kw)
    if t_mixed <= tau:
        return dict(mode=AGG, s_p=total, s_d=0, k=1, rho=None, t=t_mixed, flags=0)
    pre, dec = split_requests(batch)
    t_decode_tokens = len(dec)
    t_prefill_tokens = sum(q for q, _ in pre)
    best_rho, best = 0.0, None
    for s_d in range(step, total, step):
        t_d = f_roofline(dec, s_d, tables, kinds={1} if dec else (), **kw)
        if t_d > tau:
            continue
        s_p = total - s_d
        t_p = f_roofline(pre, s_p, tables, kinds={0} if pre else (), **kw)
        base = math.floor(t_p / t_d) if t_d > 0 else 1
        # rho(k) rises up to k = base and falls from k = base + 1 on, so under a cap on the
        # decode steps the best allowed candidates are base and base + 1 clamped to the cap
        cands = (base, base + 1) if kmax is None else tuple(sorted({min(base, kmax), min(base + 1, kmax)}))
        for k in cands:
            if k < 1:
                continue
            t = max(k * t_d, t_p)
            rho = (k * t_decode_tokens + t_prefill_tokens) / t
            if rho > best_rho:
                best_rho, best = rho, dict(mode=SPLIT, s_p=s_p, s_d=s_d, k=k, rho=rho, t=t, flags=0)
    if best is None:
        return dict(mode=AGG, s_p=total, s_d=0, k=1, rho=None, t=t_mixed, flags=SLO_INFEASIBLE)
    return best


# ---- full-model estimate (token-level operators, Section 4.1) ---------------------------------

@dataclass
class Block:
    """Dense dimensions of a transformer block: FFN width m and the classifier's vocabulary."""
    ffn_dim: int
    vocab_size: int = 0
    gqa_qkv: bool = False      # QKV output width (h_q + 2 h_kv) d_h instead of the paper's d
    fused_gate_up: bool = False  # gate-up output width 2 m instead of m


def linear_cost(n, d_i, d_o, b):
    """(F_lin, B_lin) of n tokens through a d_i x d_o linear operator."""
    return 2.0 * n * d_i * d_o, n * d_i * b + d_i * d_o * b + n * d_o * b


def rmsnorm_cost(n, d, b):
    """Reading: square, sum, scale and weight per element; read x, write y, read the weight."""
    return 4.0 * n * d, 2.0 * n * d * b + d * b


def swiglu_cost(n, m, b):
    """Reading: silu(gate) * up, about five operations per element; read gate and up, write."""
    return 5.0 * n * m, 3.0 * n * m * b


def add_cost(n, d, b):
    """Residual add: one operation per element; read two tensors, write one."""
    return 1.0 * n * d, 3.0 * n * d * b


def token_ops(n, block, *, h_q, h_kv, d_h, b):
    """(F, B) of each token-level operator of one layer for n tokens, in block order."""
    d = h_q * d_h
    m = block.ffn_dim
    d_qkv = (h_q + 2 * h_kv) * d_h if block.gqa_qkv else d
    m_gu = 2 * m if block.fused_gate_up else m
    return [rmsnorm_cost(n, d, b), linear_cost(n, d, d_qkv, b), linear_cost(n, d, d, b), add_cost(n, d, b),
            rmsnorm_cost(n, d, b), linear_cost(n, d, m_gu, b), swiglu_cost(n, m, b), linear_cost(n, m, d, b),
            add_cost(n, d, b)]


def t_tok(n, s, tables, block, *, h_q, h_kv, d_h, b):
    """Seconds for one layer's token-level operators on n tokens and s CUs (none for n = 0)."""
    if n == 0:
        return 0.0
    pi, bw = tables.pi(s), tables.b(s)
    return sum(max(f / pi, by / bw) for f, by in token_ops(n, block, h_q=h_q, h_kv=h_kv, d_h=d_h, b=b))


def t_cls(n_rows, s, tables, block, *, h_q, d_h, b):
    """Seconds for the classifier (d -> vocab_size) on n_rows rows."""
    if n_rows == 0 or block.vocab_size == 0:
        return 0.0
    f, by = linear_cost(n_rows, h_q * d_h, block.vocab_size, b)
    return max(f / tables.pi(s), by / tables.b(s))


def f_model(reqs, s, tables, block, *, h_q, h_kv, d_h, b, layers, kinds=()) -> float:
    """t_total = L (t_tok + t_attn) + t_cls for the requests [(q, c), ...] on s CUs."""
    n = sum(q for q, _ in reqs)
    per_layer = t_tok(n, s, tables, block, h_q=h_q, h_kv=h_kv, d_h=d_h, b=b) + \
        t_attn(reqs, s, tables, h_q, h_kv, d_h, b) + tables.launch(kinds, s)
    return layers * per_layer + t_cls(len(reqs), s, tables, block, h_q=h_q, d_h=d_h, b=b)


def predict_model(batch, mode, s_p, s_d, k, tables, block, *, h_q, h_kv, d_h, b, layers, total=TOTAL_CUS) -> float:
    """Full-model iteration latency in seconds: aggregated, or max(k t_d(S_d), t_p(S_p)) where each
    partition runs all layers for its own tokens."""
    kw = dict(h_q=h_q, h_kv=h_kv, d_h=d_h, b=b, layers=layers)
    if mode == AGG:
        return f_model([(q, c) for _, q, c in batch], total, tables, block, kinds=kinds_of(batch), **kw)
    pre, dec = split_requests(batch)
    t_d = f_model(dec, s_d, tables, block, kinds={1} if dec else (), **kw)
    t_p = f_model(pre, s_p, tables, block, kinds={0} if pre else (), **kw)
    return max(k * t_d, t_p)


def choose_model(batch, tau, tables, block, *, h_q, h_kv, d_h, b, layers, total=TOTAL_CUS, step=SPLIT_STEP,
                 kmax=None):
    """Algorithm 1 on the full-model estimate (same steps as choose)."""
    kw = dict(h_q=h_q, h_kv=h_kv, d_h=d_h, b=b, layers=layers)
    t_mixed = f_model([(q, c) for _, q, c in batch], total, tables, block, kinds=kinds_of(batch), **kw)
    if t_mixed <= tau:
        return dict(mode=AGG, s_p=total, s_d=0, k=1, rho=None, t=t_mixed, flags=0)
    pre, dec = split_requests(batch)
    t_decode_tokens = len(dec)
    t_prefill_tokens = sum(q for q, _ in pre)
    best_rho, best = 0.0, None
    for s_d in range(step, total, step):
        t_d = f_model(dec, s_d, tables, block, kinds={1} if dec else (), **kw)
        if t_d > tau:
            continue
        s_p = total - s_d
        t_p = f_model(pre, s_p, tables, block, kinds={0} if pre else (), **kw)
        base = math.floor(t_p / t_d) if t_d > 0 else 1
        cands = (base, base + 1) if kmax is None else tuple(sorted({min(base, kmax), min(base + 1, kmax)}))
        for k in cands:
            if k < 1:
                continue
            t = max(k * t_d, t_p)
            rho = (k * t_decode_tokens + t_prefill_tokens) / t
            if rho > best_rho:
                best_rho, best = rho, dict(mode=SPLIT, s_p=s_p, s_d=s_d, k=k, rho=rho, t=t, flags=0)
    if best is None:
        return dict(mode=AGG, s_p=total, s_d=0, k=1, rho=None, t=t_mixed, flags=SLO_INFEASIBLE)
    return best
