"""Seeded synthetic inputs shaped like the long-context workloads of the DLA paper.

This module only draws random numbers; it contains none of the method's
arithmetic, so both the HIP path and the float64 oracle can take their inputs
from it.  Everything is drawn in float64 from numpy PCG64 streams keyed by
(seed, sequence, head, stream-id) -- any (b, h) slice can be regenerated on its
own -- and then rounded to the storage dtype (float32, or bfloat16 by
round-to-nearest-even of the float32 value).  Consumers that need exact values
of what is stored use :func:`to_f64`.

Token model (piecewise-stationary, the setting of the paper's corollary on
fixed blocking, Sec. 3.1):

* segment boundaries are shared by all heads of a sequence;
* every (head, segment) draws means mu_k, mu_v ~ N(0, I);
* a token of a segment with correlation rho2 has
  k = normalise(sqrt(rho2) mu_k + sqrt(1 - rho2) e),  v = sqrt(rho2) mu_v + sqrt(1 - rho2) e'
  (v is marginally N(0, I) exactly), q = normalise(N(0, I));
* log-decay gates g ~ U(g_lo, 0) i.i.d. per (b, h, t);
* readout weights lambda[t, j] = 1 + 0.5 (w_j . q_t) with w_j ~ N(0, I) per
  (head, slot): a linear layer over the query, as Sec. 3.2 describes.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

# Stream ids used as the last word of the RNG key.
_S_SEG, _S_MU, _S_K, _S_V, _S_Q, _S_G, _S_W, _S_BETA = range(8)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    T: int
    dk: int
    dv: int
    C: int
    tau: float
    dtype: str            # "f32" or "bf16": storage type of q, k, v, lambda and o
    g_lo: float
    seed: int
    structure: str        # "cuts" | "geom" | "spans_bursts" | "iid"
    n_seg: int = 0        # "cuts": number of segments
    mean_len: float = 64  # "geom": mean segment length
    rho2: float = 0.95
    span_mean: float = 1024.0
    burst_mean: float = 16.0
    rho2_span: float = 0.98
    decode_steps: int = 0  # decode workloads: i.i.d. tokens after the prefix

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def label(self) -> str:
        return (f"{self.name}: B{self.B} H{self.H} T{self.T} dk{self.dk} dv{self.dv} "
                f"C{self.C} tau{self.tau} {self.dtype}")


WORKLOADS = {
    # fp32 correctness case, 6 planted segments
    "cfg1": Workload("cfg1", 1, 2, 512, 64, 64, 8, 0.5, "f32", -0.05, 1, "cuts", n_seg=6),
    # literal i.i.d. variant of cfg1: every token opens a state, merges every step
    "cfg1_iid": Workload("cfg1_iid", 1, 2, 512, 64, 64, 8, 0.5, "f32", -0.05, 1, "iid"),
    # 64 segments of geometric length (mean 64)
    "cfg2": Workload("cfg2", 8, 16, 4096, 128, 128, 64, 0.5, "bf16", -0.05, 2, "geom", mean_len=64),
    # long stable spans (~1k tokens) alternating with short i.i.d. bursts (~16 tokens)
    "cfg3": Workload("cfg3", 4, 16, 16384, 128, 128, 128, 0.5, "bf16", -0.05, 3, "spans_bursts"),
    # long-context prefill, 1024 segments, slow decay
    "cfg4": Workload("cfg4", 1, 32, 65536, 128, 128, 256, 0.5, "bf16", -0.01, 4, "cuts", n_seg=1024),
    # decode: 32k-token geometric-segment prefix, then i.i.d. decode tokens
    "cfg5": Workload("cfg5", 64, 32, 32768, 128, 128, 128, 0.5, "bf16", -0.05, 5, "geom",
                     mean_len=64, decode_steps=256),
}


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *key])))


# ----------------------------------------------------------------------------
# dtype helpers
# ----------------------------------------------------------------------------

def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float64/float32 -> bfloat16 bit patterns (uint16): x is first rounded to
    float32, then to bfloat16 with round-to-nearest-even."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> 16) & 1
    r = (b + np.uint32(0x7FFF) + lsb) >> 16
    return r.astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the storage dtype."""
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return round_to_bf16_bits(x)
    raise ValueError(dtype)


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of a stored array."""
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    return np.asarray(a, dtype=np.float64)


# ----------------------------------------------------------------------------
# segment structure
# ----------------------------------------------------------------------------

def segment_plan(w: Workload, b: int, T: Optional[int] = None):
    """Per-token segment id and per-token rho2 for sequence b.

    Returns (seg_id[T] int64, rho2[T] float64).  Tokens of an i.i.d. burst get
    rho2 = 0 and a segment id of their own."""
    T = w.T if T is None else T
    rng = _rng(w.seed, b, 0, _S_SEG)
    if w.structure == "iid":
        return np.arange(T, dtype=np.int64), np.zeros(T)
    if w.structure == "cuts":
        n_cut = min(max(w.n_seg - 1, 0), T - 1)
        cuts = np.sort(rng.choice(np.arange(1, T), size=n_cut, replace=False))
        seg = np.zeros(T, dtype=np.int64)
        seg[cuts] = 1
        return np.cumsum(seg), np.full(T, w.rho2)
    if w.structure == "geom":
        lens = []
        tot = 0
        while tot < T:
            L = int(rng.geometric(1.0 / w.mean_len))
            lens.append(L)
            tot += L
        seg = np.repeat(np.arange(len(lens), dtype=np.int64), lens)[:T]
        return seg, np.full(T, w.rho2)
    if w.structure == "spans_bursts":
        seg = np.empty(T, dtype=np.int64)
        rho = np.empty(T)
        t = 0
        sid = 0
        stable = True
        while t < T:
            if stable:
                L = int(rng.geometric(1.0 / w.span_mean))
                e = min(T, t + L)
                seg[t:e] = sid
                rho[t:e] = w.rho2_span
                sid += 1
            else:
                L = int(rng.geometric(1.0 / w.burst_mean))
                e = min(T, t + L)
                n = e - t
                seg[t:e] = sid + np.arange(n)
                rho[t:e] = 0.0
                sid += n
            t = e
            stable = not stable
        return seg, rho
    raise ValueError(w.structure)


def _head_tokens(w: Workload, b: int, h: int, seg: np.ndarray, rho2: np.ndarray,
                 t0: int = 0):
    """k, v, q, g (float64) for one head, tokens t0 .. t0+len(seg)-1."""
    T = len(seg)
    nseg = int(seg.max()) + 1 if T else 0
    mu = _rng(w.seed, b, h, _S_MU)
    mu_k = mu.standard_normal((nseg, w.dk))
    mu_v = mu.standard_normal((nseg, w.dv))
    a = np.sqrt(rho2)[:, None]
    c = np.sqrt(1.0 - rho2)[:, None]
    ek = _rng(w.seed, b, h, _S_K, t0).standard_normal((T, w.dk))
    ev = _rng(w.seed, b, h, _S_V, t0).standard_normal((T, w.dv))
    k = a * mu_k[seg] + c * ek
    k /= np.linalg.norm(k, axis=1, keepdims=True)
    v = a * mu_v[seg] + c * ev
    q = _rng(w.seed, b, h, _S_Q, t0).standard_normal((T, w.dk))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    g = _rng(w.seed, b, h, _S_G, t0).uniform(w.g_lo, 0.0, size=T)
    return k, v, q, g


def lambda_weights(w: Workload, h: int) -> np.ndarray:
    """Per-head readout projection w_j (C x dk), shared by all sequences."""
    return _rng(w.seed, 0, h, _S_W).standard_normal((w.C, w.dk))


def make_beta(w: Workload, heads: Optional[list] = None, T: Optional[int] = None) -> np.ndarray:
    """Step sizes of the delta-rule form (a sigmoid output in the Gated DeltaNet
    backbone): beta ~ U(0.05, 1) i.i.d. per (b, h, t), float32 [n_heads, T]."""
    T = w.T if T is None else T
    if heads is None:
        heads = [(b, h) for b in range(w.B) for h in range(w.H)]
    out = np.empty((len(heads), T), np.float32)
    for i, (b, h) in enumerate(heads):
        out[i] = _rng(w.seed, b, h, _S_BETA).uniform(0.05, 1.0, size=T)
    return out


def _parallel(fn, n):
    """Run fn(i) for i < n on a thread pool (numpy releases the GIL in the bulk
    kernels used here); results are written in place, so the order is free."""
    import concurrent.futures as cf
    import os
    workers = max(1, min(n, int(os.environ.get("DLA_GEN_THREADS", os.cpu_count() or 1)), 16))
    if workers == 1:
        for i in range(n):
            fn(i)
        return
    with cf.ThreadPoolExecutor(workers) as ex:
        list(ex.map(fn, range(n)))


def make_inputs(w: Workload, heads: Optional[list] = None, with_lambda: bool = True,
                with_q: bool = True):
    """Draw the inputs of a prefill workload.

    heads: optional list of (b, h) pairs; default all B*H heads.  Returns a dict
    with stored arrays q, k, v, lam ([n_heads, T, *]) in the storage dtype,
    g ([n_heads, T] float32), and 'heads'.  Arrays are laid out [B*H, T, d]
    (equivalently [B, H, T, d] when all heads are drawn)."""
    if heads is None:
        heads = [(b, h) for b in range(w.B) for h in range(w.H)]
    n = len(heads)
    sdt = np.float32 if w.dtype == "f32" else np.uint16
    out = {
        "k": np.empty((n, w.T, w.dk), sdt),
        "v": np.empty((n, w.T, w.dv), sdt),
        "g": np.empty((n, w.T), np.float32),
        "heads": list(heads),
    }
    if with_q:
        out["q"] = np.empty((n, w.T, w.dk), sdt)
    if with_lambda:
        out["lam"] = np.empty((n, w.T, w.C), sdt)
    plans = {b: segment_plan(w, b) for b in sorted({b for b, _ in heads})}

    def one(i):
        b, h = heads[i]
        seg, rho2 = plans[b]
        k, v, q, g = _head_tokens(w, b, h, seg, rho2)
        out["k"][i] = store(k, w.dtype)
        out["v"][i] = store(v, w.dtype)
        out["g"][i] = g.astype(np.float32)
        if with_q:
            out["q"][i] = store(q, w.dtype)
        if with_lambda:
            # lambda is drawn from the stored (rounded) query, as a layer would see it
            qs = to_f64(out["q"][i], w.dtype) if with_q else q
            out["lam"][i] = store(1.0 + 0.5 * (qs @ lambda_weights(w, h).T), w.dtype)

    _parallel(one, n)
    return out


def make_decode_tokens(w: Workload, steps: Optional[int] = None, heads: Optional[list] = None):
    """i.i.d. decode tokens (rho2 = 0) following a prefix of w.T tokens:
    arrays [n_heads, steps, *]."""
    steps = w.decode_steps if steps is None else steps
    if heads is None:
        heads = [(b, h) for b in range(w.B) for h in range(w.H)]
    n = len(heads)
    sdt = np.float32 if w.dtype == "f32" else np.uint16
    out = {k: np.empty((n, steps, d), sdt) for k, d in (("q", w.dk), ("k", w.dk), ("v", w.dv))}
    out["g"] = np.empty((n, steps), np.float32)
    out["lam"] = np.empty((n, steps, w.C), sdt)
    seg = np.arange(steps, dtype=np.int64)
    rho2 = np.zeros(steps)

    def one(i):
        b, h = heads[i]
        k, v, q, g = _head_tokens(w, b, h, seg, rho2, t0=w.T)
        out["k"][i] = store(k, w.dtype)
        out["v"][i] = store(v, w.dtype)
        out["q"][i] = store(q, w.dtype)
        out["g"][i] = g.astype(np.float32)
        out["lam"][i] = store(1.0 + 0.5 * (to_f64(out["q"][i], w.dtype) @ lambda_weights(w, h).T),
                              w.dtype)

    _parallel(one, n)
    out["heads"] = list(heads)
    return out


def make_prefix_torch(w: Workload, device, with_q: bool = False, with_lambda: bool = False):
    """Device-side draw of a prefill workload's k, v, g (and q, lambda) with
    the same recipe as make_inputs, from torch's generator seeded with w.seed:
    for prefixes too large to draw on the host (B*H*T in the billions).  Values
    differ from make_inputs' numpy streams; the segment plan is the same.
    Returns bf16/f32 tensors q, k [B, H, T, d_k], v [B, H, T, d_v], g [B, H, T]
    float32, and with with_lambda (which implies with_q) lam [B, H, T, C]."""
    with_q = with_q or with_lambda
    import torch
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    gen = torch.Generator(device=device)
    gen.manual_seed(int(w.seed) * 1000003 + 17)
    k = torch.empty((w.B, w.H, w.T, w.dk), dtype=tdt, device=device)
    v = torch.empty((w.B, w.H, w.T, w.dv), dtype=tdt, device=device)
    q = torch.empty((w.B, w.H, w.T, w.dk), dtype=tdt, device=device) if with_q else None
    g = torch.empty((w.B, w.H, w.T), dtype=torch.float32, device=device)
    for b in range(w.B):
        seg_np, rho_np = segment_plan(w, b)
        seg = torch.from_numpy(seg_np).to(device)
        a = torch.from_numpy(np.sqrt(rho_np)).to(device=device, dtype=torch.float32)[None, :, None]
        c = torch.from_numpy(np.sqrt(1.0 - rho_np)).to(device=device,
                                                     dtype=torch.float32)[None, :, None]
        nseg = int(seg_np.max()) + 1
        mu_k = torch.randn((w.H, nseg, w.dk), generator=gen, device=device)
        mu_v = torch.randn((w.H, nseg, w.dv), generator=gen, device=device)
        kk = a * mu_k[:, seg] + c * torch.randn((w.H, w.T, w.dk), generator=gen, device=device)
        k[b] = (kk / kk.norm(dim=-1, keepdim=True)).to(tdt)
        v[b] = (a * mu_v[:, seg] + c * torch.randn((w.H, w.T, w.dv), generator=gen,
                                                   device=device)).to(tdt)
        g[b] = torch.rand((w.H, w.T), generator=gen, device=device) * w.g_lo
        if with_q:
            qq = torch.randn((w.H, w.T, w.dk), generator=gen, device=device)
            q[b] = (qq / qq.norm(dim=-1, keepdim=True)).to(tdt)
    if not with_lambda:
        return q, k, v, g
    Wt = torch.from_numpy(np.stack([lambda_weights(w, h).T for h in range(w.H)])).to(
        device=device, dtype=torch.float32).contiguous()          # [H, d_k, C]
    lam = torch.empty((w.B, w.H, w.T, w.C), dtype=tdt, device=device)
    for b in range(w.B):
        lam[b] = (1.0 + 0.5 * torch.matmul(q[b].float(), Wt)).to(tdt)
    return q, k, v, g, lam


def make_decode_tokens_torch(w: Workload, steps: int, device):
    """Device-side draw of i.i.d. decode tokens (rho2 = 0) with the recipe of
    make_decode_tokens, from torch's generator seeded with w.seed: q, k
    normalised, v ~ N(0, I), g ~ U(g_lo, 0), lambda = 1 + 0.5 (w_j . q) with the
    per-head projection of lambda_weights, computed from the stored query.
    Values differ from make_decode_tokens' numpy streams.  Returns tensors laid
    out [steps, B, H, *] (one contiguous slice per step): q, k [.., d_k], v
    [.., d_v], lam [.., C] in the storage dtype, g [steps, B, H] float32."""
    import torch
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    gen = torch.Generator(device=device)
    gen.manual_seed(int(w.seed) * 1000003 + 29)
    shp = (steps, w.B, w.H)
    q = torch.randn(shp + (w.dk,), generator=gen, device=device)
    q = (q / q.norm(dim=-1, keepdim=True)).to(tdt)
    k = torch.randn(shp + (w.dk,), generator=gen, device=device)
    k = (k / k.norm(dim=-1, keepdim=True)).to(tdt)
    v = torch.randn(shp + (w.dv,), generator=gen, device=device).to(tdt)
    g = torch.rand(shp, generator=gen, device=device) * w.g_lo
    Wt = torch.from_numpy(np.stack([lambda_weights(w, h).T for h in range(w.H)])).to(
        device=device, dtype=torch.float32).contiguous()          # [H, d_k, C]
    lam = 1.0 + 0.5 * torch.matmul(q.float().unsqueeze(-2), Wt).squeeze(-2)
    return q, k, v, g.contiguous(), lam.to(tdt).contiguous()
