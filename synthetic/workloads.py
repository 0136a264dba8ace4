"""Seeded synthetic inputs shaped like the paper's VLM workloads.

This module only draws random numbers and lays them out; it holds none of the
pruning method's arithmetic.  Both the CPU oracle side of the tests and the GPU
side read the arrays it returns.  Float inputs come back in storage form:
float32 arrays, or the uint16 bit patterns of bfloat16 (round to nearest even
from float32).

Shapes follow the models the paper evaluates (Sec. 5.1): LLaVA-1.5-7B with
576 visual tokens, LLaVA-NeXT-7B with 2,880 (5 tiles of 576), and
Qwen2.5-VL-7B-shaped inputs with 16,384 visual tokens (the sequence length the
introduction cites for Qwen2.5-VL).  Stage-1 planted structure: a few salient
patches whose [CLS] logits are raised by +4 in every head, and query-matched
patches whose feature has cosine exactly 0.6 to the mean text direction.
Stage-2 planted structure: per-head query scales from 0.5 to 2 (distinct head
variances), and a quarter of the query heads that see a shared direction in a
set of "relevant" visual key rows (a +3 logit boost).
"""

import math
from dataclasses import dataclass, field, replace

import numpy as np

PREFIX_LEN = 35  # stand-in chat-template prefix before the visual block


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    N: int
    n_seg: int
    H_v: int
    d: int            # projected width d'
    M_max: int        # padded text rows
    K1: int
    K2: int
    H_q: int
    H_kv: int
    d_h: int
    D: int            # LLM hidden size
    n_keep: int       # |H*|
    n_pos: int        # 1, or 3 for M-RoPE position ids
    dtype: str        # "f32" | "bf16"
    n_sal: int
    n_qm: int
    text_len: tuple = ("fixed",)   # ("fixed",) = M_max, or ("uniform", lo, hi)
    rho: float = 0.5
    qm_blocks: int = 0             # >0: query-matched tokens in square blocks on a grid
    grid: int = 0                  # side of the token grid (for blocks and M-RoPE)
    P: int = PREFIX_LEN
    seed: int = 0
    tie_stress: bool = False
    extra: dict = field(default_factory=dict)

    @property
    def T_max(self):
        return self.M_max

    @property
    def S(self):
        return self.P + self.K1 + self.T_max

    @property
    def S_out(self):
        return self.P + self.K2 + self.T_max

    @property
    def elem_bytes(self):
        return 4 if self.dtype == "f32" else 2

    def with_(self, **kw):
        return replace(self, **kw)


WORKLOADS = {
    # LLaVA-1.5-7B shapes, batch 1, fp32
    "llava15-b1-f32": Workload(
        "llava15-b1-f32", B=1, N=576, n_seg=1, H_v=16, d=4096, M_max=32,
        K1=192, K2=32, H_q=32, H_kv=32, d_h=128, D=4096, n_keep=8, n_pos=1,
        dtype="f32", n_sal=8, n_qm=10, grid=24, seed=1000),
    # LLaVA-1.5-7B shapes, batch 64, bf16, text length uniform in [16, 64]
    "llava15-b64-bf16": Workload(
        "llava15-b64-bf16", B=64, N=576, n_seg=1, H_v=16, d=4096, M_max=64,
        K1=192, K2=64, H_q=32, H_kv=32, d_h=128, D=4096, n_keep=16, n_pos=1,
        dtype="bf16", n_sal=8, n_qm=10, text_len=("uniform", 16, 64), grid=24,
        seed=2000),
    # LLaVA-NeXT-7B shapes, batch 16, 5 tiles x 576 tokens
    "llavanext-b16-bf16": Workload(
        "llavanext-b16-bf16", B=16, N=2880, n_seg=5, H_v=16, d=4096, M_max=64,
        K1=640, K2=160, H_q=32, H_kv=32, d_h=128, D=4096, n_keep=16, n_pos=1,
        dtype="bf16", n_sal=24, n_qm=40, grid=24, seed=3000),
    # Qwen2.5-VL-7B shapes, batch 4, 16,384 visual tokens, GQA 28/4, M-RoPE
    "qwen25vl-b4-bf16": Workload(
        "qwen25vl-b4-bf16", B=4, N=16384, n_seg=1, H_v=16, d=3584, M_max=128,
        K1=4096, K2=1024, H_q=28, H_kv=4, d_h=128, D=3584, n_keep=14, n_pos=3,
        dtype="bf16", n_sal=228, n_qm=256, qm_blocks=4, grid=128, seed=4000),
    # Sweep base: LLaVA-1.5 shapes, batch 32 (K1/K2/n_keep/rho varied by sweep())
    "sweep-llava15-b32-bf16": Workload(
        "sweep-llava15-b32-bf16", B=32, N=576, n_seg=1, H_v=16, d=4096,
        M_max=32, K1=144, K2=48, H_q=32, H_kv=32, d_h=128, D=4096, n_keep=8,
        n_pos=1, dtype="bf16", n_sal=8, n_qm=10, grid=24, seed=5000),
}

DEFAULT_BENCH_WORKLOAD = "qwen25vl-b4-bf16"


def keep_count(ratio, n):
    """floor(ratio * n + 1/2) clamped to [1, n] (budget bookkeeping)."""
    return int(min(max(math.floor(ratio * n + 0.5), 1), n))


def sweep():
    """The sweep grid: keep ratio x textual ratio x head count, K1:K2 = 3:1."""
    base = WORKLOADS["sweep-llava15-b32-bf16"]
    out = []
    for r in (0.5, 0.25, 1 / 9, 1 / 18):
        k1 = keep_count(r, base.N)
        k2 = keep_count(1 / 3, k1)
        for rho in (0.0, 0.25, 0.5, 0.75, 1.0):
            for nk in (4, 8, 16, 32):
                out.append(base.with_(K1=k1, K2=k2, rho=rho, n_keep=nk))
    return out


# ----------------------------------------------------------------------------
# storage conversion
# ----------------------------------------------------------------------------


def to_storage(x, dtype):
    """float64/float32 -> float32, or -> bfloat16 bit patterns (uint16) by
    rounding the float32 value to nearest even."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f32":
        return f
    u = f.view(np.uint32).copy()
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    u += np.uint32(0x7FFF)
    u += lsb
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def _rng(w, stage, b):
    return np.random.default_rng([w.seed, stage, b])


def _text_lengths(w):
    if w.text_len[0] == "fixed":
        return np.full(w.B, w.M_max, dtype=np.int32)
    _, lo, hi = w.text_len
    rng = np.random.default_rng([w.seed, 9])
    return rng.integers(lo, hi + 1, size=w.B).astype(np.int32)


def _block_tokens(rng, grid, n_blocks, n_tokens):
    """n_tokens tokens in n_blocks square blocks on a grid x grid token map,
    blocks placed at random, non-overlapping."""
    side = int(round(math.sqrt(n_tokens / n_blocks)))
    cells = grid // side
    picks = rng.choice(cells * cells, size=n_blocks, replace=False)
    toks = []
    for c in picks:
        r0, c0 = (c // cells) * side, (c % cells) * side
        for r in range(side):
            for cc in range(side):
                toks.append((r0 + r) * grid + c0 + cc)
    return np.array(sorted(toks), dtype=np.int64)


def stage1_inputs(w):
    """Stage-1 inputs for every sample of workload w.

    Returns dict: cls_logits [B,H_v,N], vis_feats [B,N,d], text_emb
    [B,M_max,d] (rows >= text_len are zero), text_len int32 [B], and the
    planted index sets (salient, matched) per sample."""
    B, N, d, H = w.B, w.N, w.d, w.H_v
    lens = _text_lengths(w)
    cls = np.empty((B, H, N), dtype=np.float32 if w.dtype == "f32" else np.uint16)
    Zs = np.empty((B, N, d), dtype=cls.dtype)
    Ts = np.zeros((B, w.M_max, d), dtype=cls.dtype)
    sal_sets, qm_sets = [], []
    for b in range(B):
        rng = _rng(w, 1, b)
        if w.qm_blocks:
            qm = _block_tokens(rng, w.grid, w.qm_blocks, w.n_qm)
        else:
            qm = np.sort(rng.choice(N, size=w.n_qm, replace=False))
        rest = np.setdiff1d(np.arange(N), qm)
        sal = np.sort(rng.choice(rest, size=w.n_sal, replace=False))
        L = rng.standard_normal((H, N))
        L[:, sal] += 4.0
        Z = rng.standard_normal((N, d), dtype=np.float32) * np.float32(1 / math.sqrt(d))
        T = rng.standard_normal((int(lens[b]), d)) / math.sqrt(d)
        u = T.mean(axis=0)
        u /= np.linalg.norm(u)
        for i in qm:
            g = rng.standard_normal(d)
            g -= (g @ u) * u
            g /= np.linalg.norm(g)
            Z[i] = np.linalg.norm(Z[i].astype(np.float64)) * (0.6 * u + 0.8 * g)
        if w.tie_stress:
            # a quarter of the tokens copy the logits column and feature row
            # of one of 64 prototype tokens
            protos = rng.choice(N, size=64, replace=False)
            others = np.setdiff1d(np.arange(N), protos)
            copies = rng.choice(others, size=N // 4, replace=False)
            src = protos[rng.integers(0, 64, size=copies.size)]
            L[:, copies] = L[:, src]
            Z[copies] = Z[src]
        cls[b] = to_storage(L, w.dtype)
        Zs[b] = to_storage(Z, w.dtype)
        Ts[b, :lens[b]] = to_storage(T, w.dtype)
        sal_sets.append(sal)
        qm_sets.append(qm)
    return dict(cls_logits=cls, vis_feats=Zs, text_emb=Ts, text_len=lens,
                salient=sal_sets, matched=qm_sets)


def _positions(w, kept_vis):
    """Position ids [n_pos, S] for one sample: arange for 1-D RoPE; for the
    3-row M-RoPE layout prefix/text tokens get (p, p, p) and visual token j
    gets (P, P + row, P + col) of its original grid cell."""
    S, P, K1 = w.S, w.P, w.K1
    if w.n_pos == 1:
        return np.arange(S, dtype=np.int64)[None]
    pos = np.empty((3, S), dtype=np.int64)
    pos[:, :P] = np.arange(P)
    grid = w.grid if w.grid else int(math.isqrt(w.N))
    rows, cols = np.divmod(kept_vis, grid)
    pos[0, P:P + K1] = P
    pos[1, P:P + K1] = P + rows
    pos[2, P:P + K1] = P + cols
    start = P + grid
    pos[:, P + K1:] = start + np.arange(w.T_max)
    return pos


def stage2_inputs(w, with_lse_rest=False):
    """Stage-2 inputs at the pruning layer for every sample of workload w.

    Sequence layout [prefix P | K1 visual | T_max text].  Returns dict: q
    [B,S,H_q,d_h], k and v [B,S,H_kv,d_h], hidden [B,S,D], pos int64
    [n_pos,B,S], text_len int32 [B], optionally lse_rest float32 [B,H_q,T_max],
    and the planted relevant visual rows and sensitive heads per sample.
    With tie_stress a quarter of the visual key rows are copies of prototype
    rows (exact ties in the token score)."""
    B, S, Hq, Hkv, dh, D = w.B, w.S, w.H_q, w.H_kv, w.d_h, w.D
    G = Hq // Hkv
    lens = _text_lengths(w)
    sd = np.float32 if w.dtype == "f32" else np.uint16
    q = np.empty((B, S, Hq, dh), dtype=sd)
    k = np.empty((B, S, Hkv, dh), dtype=sd)
    v = np.empty((B, S, Hkv, dh), dtype=sd)
    hidden = np.empty((B, S, w.D), dtype=sd)
    pos = np.empty((w.n_pos, B, S), dtype=np.int64)
    lse_rest = np.empty((B, Hq, w.T_max), dtype=np.float32) if with_lse_rest else None
    rel_sets, sens_sets = [], []
    a = math.sqrt(3.0 * math.sqrt(dh))
    for b in range(B):
        rng = _rng(w, 2, b)
        beta = rng.permutation(np.linspace(0.5, 2.0, Hq))
        Q = rng.standard_normal((S, Hq, dh), dtype=np.float32) * beta[None, :, None].astype(np.float32)
        Kt = rng.standard_normal((S, Hkv, dh), dtype=np.float32)
        Vt = rng.standard_normal((S, Hkv, dh), dtype=np.float32)
        Hd = rng.standard_normal((S, D), dtype=np.float32)
        sens = np.sort(rng.choice(Hq, size=max(1, Hq // 4), replace=False))
        n_rel = max(1, w.K2 // 2)
        rel = np.sort(rng.choice(w.K1, size=n_rel, replace=False))
        c = rng.standard_normal((Hkv, dh))
        c /= np.linalg.norm(c, axis=1, keepdims=True)
        for g in range(Hkv):
            Kt[w.P + rel, g, :] += (a * c[g]).astype(np.float32)
        for h in sens:
            Q[w.P + w.K1:, h, :] += (a * c[h // G]).astype(np.float32)
        if w.tie_stress and w.K1 >= 4:
            # a quarter of the visual key rows copy one of (up to) 64
            # prototype visual rows in every KV head: their logits, and so
            # their token scores, tie exactly
            n_proto = min(64, w.K1 // 4)
            protos = rng.choice(w.K1, size=n_proto, replace=False)
            others = np.setdiff1d(np.arange(w.K1), protos)
            copies = rng.choice(others, size=w.K1 // 4, replace=False)
            src = protos[rng.integers(0, n_proto, size=copies.size)]
            Kt[w.P + copies] = Kt[w.P + src]
        kept_vis = np.sort(rng.choice(w.N, size=w.K1, replace=False))
        q[b] = to_storage(Q, w.dtype)
        k[b] = to_storage(Kt, w.dtype)
        v[b] = to_storage(Vt, w.dtype)
        hidden[b] = to_storage(Hd, w.dtype)
        pos[:, b] = _positions(w, kept_vis)
        if with_lse_rest:
            lse_rest[b] = (rng.standard_normal((Hq, w.T_max))
                           + np.log(w.P + 1 + np.arange(w.T_max))[None, :])
        rel_sets.append(rel)
        sens_sets.append(sens)
    return dict(q=q, k=k, v=v, hidden=hidden, pos=pos, text_len=lens,
                lse_rest=lse_rest, relevant=rel_sets, sensitive=sens_sets)


def sensitivity_inputs(w, rephrase=0.1, with_lse_rest=False):
    """Two questions about one image for the text-sensitivity analysis.

    Layout per question as in stage2_inputs.  The image's key rows are shared
    by both questions (k [B,S,H_kv,d_h]); two unit directions per KV group are
    planted in two disjoint sets of visual key rows.  Question 0's query rows
    are N(0,1) scaled per head by a permutation of linspace(0.5, 2, H_q);
    question 1 repeats them plus `rephrase` * N(0,1) (a reworded question),
    except that on a quarter of the heads ("sensitive") the text rows carry
    the first direction in question 0 and the second in question 1.  Text
    lengths are drawn per question.  Returns dict: q0, q1, k, text_len0,
    text_len1, optionally lse_rest0/lse_rest1 [B,H_q,T_max], sensitive."""
    B, S, Hq, Hkv, dh = w.B, w.S, w.H_q, w.H_kv, w.d_h
    G = Hq // Hkv
    sd = np.float32 if w.dtype == "f32" else np.uint16
    q0 = np.empty((B, S, Hq, dh), dtype=sd)
    q1 = np.empty((B, S, Hq, dh), dtype=sd)
    k = np.empty((B, S, Hkv, dh), dtype=sd)
    lens0 = _text_lengths(w)
    lens1 = _text_lengths(w.with_(seed=w.seed + 17))
    lse = [np.empty((B, Hq, w.T_max), dtype=np.float32) for _ in range(2)] if with_lse_rest else None
    sens_sets = []
    a = math.sqrt(3.0 * math.sqrt(dh))
    T0 = w.P + w.K1
    for b in range(B):
        rng = _rng(w, 3, b)
        beta = rng.permutation(np.linspace(0.5, 2.0, Hq)).astype(np.float32)
        Q = rng.standard_normal((S, Hq, dh), dtype=np.float32) * beta[None, :, None]
        Q1 = Q + np.float32(rephrase) * rng.standard_normal((S, Hq, dh), dtype=np.float32)
        Kt = rng.standard_normal((S, Hkv, dh), dtype=np.float32)
        sens = np.sort(rng.choice(Hq, size=max(1, Hq // 4), replace=False))
        n_rel = min(max(1, w.K1 // 8), w.K1 // 2)  # none when there is a single visual row
        rows = rng.choice(w.K1, size=2 * n_rel, replace=False)
        c = rng.standard_normal((2, Hkv, dh))
        c /= np.linalg.norm(c, axis=2, keepdims=True)
        for g in range(Hkv):
            Kt[w.P + rows[:n_rel], g, :] += (a * c[0, g]).astype(np.float32)
            Kt[w.P + rows[n_rel:], g, :] += (a * c[1, g]).astype(np.float32)
        for h in sens:
            Q[T0:, h, :] += (a * c[0, h // G]).astype(np.float32)
            Q1[T0:, h, :] = Q[T0:, h, :] - (a * c[0, h // G]).astype(np.float32) + (a * c[1, h // G]).astype(np.float32)
        q0[b] = to_storage(Q, w.dtype)
        q1[b] = to_storage(Q1, w.dtype)
        k[b] = to_storage(Kt, w.dtype)
        if with_lse_rest:
            for c_ in range(2):
                lse[c_][b] = (rng.standard_normal((Hq, w.T_max))
                              + np.log(w.P + 1 + np.arange(w.T_max))[None, :])
        sens_sets.append(sens)
    return dict(q0=q0, q1=q1, k=k, text_len0=lens0, text_len1=lens1,
                lse_rest0=None if lse is None else lse[0], lse_rest1=None if lse is None else lse[1],
                sensitive=sens_sets)
