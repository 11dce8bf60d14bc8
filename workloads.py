"""Seeded synthetic workloads for the MoE expert layer (forward + backward).

This module only *draws inputs*.  It holds none of the layer's arithmetic: no
router logits, no top-k selection of real tokens, no permutation, no expert
math.  Both the HIP path and the CPU oracle consume what it returns.

The paper (Mixture-of-Parallelisms, Sec. 3.1 notation: H model width, E
experts, I per-expert intermediate width, k top-k degree, N tokens per device)
prints no model shapes and names no dataset, so every workload here is a
synthetic stand-in with the shapes below (d = H, f = I, T = N):

  tiny        T=256    d=128  E=8    k=2  f=256   near-uniform routing
  mid         T=4096   d=2048 E=64   k=6  f=1408  near-uniform routing
  large_skew  T=8192   d=4096 E=128  k=8  f=1536  router bias -> Zipf(1.2) load,
                                                  capped at T, 8 empty experts
  ep_share    T=16384  d=7168 E=384  k=8  f=2048  32 local experts [0, 32)
  long        T=65536  d=4096 E=128  k=8  f=1536  8 hot experts take 50 %

Distributions: x, dy ~ N(0,1) rounded to bf16 (RNE); W_gate, W_up, W_down ~
N(0, 0.02) bf16; router W_r ~ N(0, 0.02) fp32.  Draw order is fixed:
x, W_r, W_gate, W_up, W_down, dy (one torch generator seeded with `seed`).

Load shaping.  A router bias b[e] is added to the logits before selection and
softmax.  It is calibrated *without* the router: the logit of expert e for a
random token x ~ N(0, I) is N(0, |W_r[:, e]|^2), so the calibration draws
independent Gaussian logits with that spread (its own numpy stream), adds the
bias and counts top-k hits.  The realised histogram of the actual router is
whatever the router produces with this bias; callers report it.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

W_STD = 0.02
FORCED_EMPTY_BIAS = -1.0e4


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    T: int
    d: int
    E: int
    k: int
    f: int
    expert_begin: int = 0
    num_local: int | None = None      # None -> all E experts are local
    routing: str = "uniform"          # uniform | zipf | hot
    zipf_s: float = 1.2
    n_empty: int = 0
    hot_n: int = 8
    hot_share: float = 0.5
    renorm: int = 0

    @property
    def E_loc(self) -> int:
        return self.E if self.num_local is None else self.num_local

    @property
    def cap(self) -> int:
        """Rows reserved for permuted buffers: T * min(k, E_loc)."""
        return self.T * min(self.k, self.E_loc)

    def describe(self) -> dict:
        out = {"workload": self.name, "T": self.T, "d": self.d, "E": self.E,
               "E_loc": self.E_loc, "k": self.k, "f": self.f,
               "routing": self.routing}
        if self.routing == "zipf":
            out.update(zipf_s=self.zipf_s, n_empty=self.n_empty)
        if self.routing == "hot":
            out.update(hot_n=self.hot_n, hot_share=self.hot_share)
        return out

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", T=256, d=128, E=8, k=2, f=256),
    "mid": Workload("mid", T=4096, d=2048, E=64, k=6, f=1408),
    "large_skew": Workload("large_skew", T=8192, d=4096, E=128, k=8, f=1536,
                           routing="zipf", zipf_s=1.2, n_empty=8),
    "ep_share": Workload("ep_share", T=16384, d=7168, E=384, k=8, f=2048,
                         expert_begin=0, num_local=32),
    "long": Workload("long", T=65536, d=4096, E=128, k=8, f=1536,
                     routing="hot", hot_n=8, hot_share=0.5),
}


def get(name_or_wl) -> Workload:
    if isinstance(name_or_wl, Workload):
        return name_or_wl
    return WORKLOADS[name_or_wl]


# --------------------------------------------------------------------------
# load shaping (router bias); independent of the router implementation
# --------------------------------------------------------------------------

def _mc_topk_counts(sigma: np.ndarray, bias: np.ndarray, k: int,
                    z: np.ndarray) -> np.ndarray:
    """Top-k hit counts of Gaussian surrogate logits z*sigma + bias."""
    logits = z * sigma[None, :] + bias[None, :]
    top = np.argpartition(-logits, k - 1, axis=1)[:, :k]
    return np.bincount(top.ravel(), minlength=bias.shape[0]).astype(np.float64)


def zipf_targets(E: int, T: int, k: int, s: float, n_empty: int) -> np.ndarray:
    """Per-rank target loads: Zipf(s) over the first E-n_empty ranks,
    water-filled so that no expert exceeds T rows and the total is T*k."""
    w = np.zeros(E)
    r = np.arange(1, E - n_empty + 1, dtype=np.float64)
    w[: E - n_empty] = r ** (-s)
    total = float(T * k)
    lo, hi = 0.0, total / w[w > 0].min() * 4.0
    for _ in range(200):
        c = 0.5 * (lo + hi)
        if np.minimum(c * w, T).sum() < total:
            lo = c
        else:
            hi = c
    return np.minimum(hi * w, T)


def calibrate_bias(wl: Workload, col_norm: np.ndarray, seed: int,
                   n_mc: int = 8192, iters: int = 120) -> np.ndarray | None:
    """Router bias [E] (fp32) shaping the expert load, or None (no bias)."""
    if wl.routing == "uniform":
        return None
    rng = np.random.Generator(np.random.PCG64(seed + 7919))
    E, k, T = wl.E, wl.k, wl.T
    sigma = col_norm.astype(np.float64)
    z = rng.standard_normal((n_mc, E))
    scale = T / n_mc
    perm = rng.permutation(E)               # rank -> expert id
    if wl.routing == "zipf":
        tgt_rank = zipf_targets(E, T, k, wl.zipf_s, wl.n_empty)
        target = np.empty(E)
        target[perm] = tgt_rank
        empty = np.zeros(E, dtype=bool)
        empty[perm[E - wl.n_empty:]] = True
        bias = np.zeros(E)
        bias[empty] = FORCED_EMPTY_BIAS
        live = ~empty
        eta = 0.3 * float(sigma.mean())
        for _ in range(iters):
            cnt = _mc_topk_counts(sigma, bias, k, z) * scale
            step = eta * (np.log(target + 0.5) - np.log(cnt + 0.5))
            bias[live] += step[live]
            bias[live] -= bias[live].mean()
        return bias.astype(np.float32)
    if wl.routing == "hot":
        hot = perm[: wl.hot_n]
        lo, hi = 0.0, 20.0 * float(sigma.mean())
        bias = np.zeros(E)
        for _ in range(60):
            beta = 0.5 * (lo + hi)
            bias[:] = 0.0
            bias[hot] = beta
            share = _mc_topk_counts(sigma, bias, k, z)[hot].sum() / (n_mc * k)
            if share < wl.hot_share:
                lo = beta
            else:
                hi = beta
        bias[:] = 0.0
        bias[hot] = 0.5 * (lo + hi)
        return bias.astype(np.float32)
    raise ValueError(f"unknown routing {wl.routing!r}")


# --------------------------------------------------------------------------
# tensor draws
# --------------------------------------------------------------------------

def _normal(shape, std, gen, device, dtype):
    t = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t.to(dtype)


def make_inputs(wl, seed: int = 0, device="cpu", with_grad: bool = True) -> dict:
    """All inputs of one forward+backward pass, as torch tensors on `device`.

    Keys: x [T,d] bf16, w_router [d,E] f32, router_bias [E] f32 or None,
    w_gate, w_up [E_loc,d,f] bf16, w_down [E_loc,f,d] bf16, dy [T,d] bf16.
    Weights exist for the local experts only.
    """
    wl = get(wl)
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    bf = torch.bfloat16
    out = {"workload": wl}
    out["x"] = _normal((wl.T, wl.d), 1.0, gen, dev, bf)
    out["w_router"] = _normal((wl.d, wl.E), W_STD, gen, dev, torch.float32)
    out["w_gate"] = _normal((wl.E_loc, wl.d, wl.f), W_STD, gen, dev, bf)
    out["w_up"] = _normal((wl.E_loc, wl.d, wl.f), W_STD, gen, dev, bf)
    out["w_down"] = _normal((wl.E_loc, wl.f, wl.d), W_STD, gen, dev, bf)
    if with_grad:
        out["dy"] = _normal((wl.T, wl.d), 1.0, gen, dev, bf)
    col_norm = out["w_router"].double().norm(dim=0).cpu().numpy()
    bias = calibrate_bias(wl, col_norm, seed)
    out["router_bias"] = None if bias is None else torch.from_numpy(bias).to(dev)
    return out


# --------------------------------------------------------------------------
# vocabulary projection (Sec. 3.4): X [N,H], W_voc [H,V], targets [N]
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class VocabWorkload:
    name: str
    N: int       # tokens on the device
    H: int       # model width
    V: int       # vocabulary size
    vblock: int  # vocabulary columns per block of the online loss

    def describe(self) -> str:
        return f"{self.name}: N={self.N} H={self.H} V={self.V} vblock={self.vblock}"


# The paper's size example is V = 2e5; the mid workload uses it with the MoE
# mid layer's N and H.  The tiny one has a ragged last block.
VOCAB_WORKLOADS = {
    "vocab_tiny": VocabWorkload("vocab_tiny", N=256, H=128, V=1000, vblock=256),
    "vocab_mid": VocabWorkload("vocab_mid", N=4096, H=2048, V=200000, vblock=16384),
}


def make_vocab_inputs(vw: VocabWorkload, seed: int = 0, device="cpu") -> dict:
    """x ~ N(0,1) bf16 [N,H]; w_voc ~ N(0, 0.02) bf16 [H,V]; target uniform
    on [0, V) int32 [N]; dloss ~ N(0,1) fp32 [N] (an arbitrary upstream
    gradient, so both signs occur).  Draw order: x, w_voc, target, dloss."""
    dev = torch.device(device)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    out = {"workload": vw}
    out["x"] = _normal((vw.N, vw.H), 1.0, gen, dev, torch.bfloat16)
    out["w_voc"] = _normal((vw.H, vw.V), W_STD, gen, dev, torch.bfloat16)
    out["target"] = torch.randint(0, vw.V, (vw.N,), generator=gen, device=dev,
                                  dtype=torch.int64).to(torch.int32)
    out["dloss"] = _normal((vw.N,), 1.0, gen, dev, torch.float32)
    return out


def make_topk(T: int, k: int, E: int, zipf_s: float, seed: int = 0) -> np.ndarray:
    """Synthetic routing (no router): for every token k distinct experts,
    drawn without replacement with probabilities proportional to
    rank^-zipf_s over a seeded random ranking of the experts (Gumbel top-k).
    Returns int32 [T, k].  zipf_s = 0 is uniform."""
    rng = np.random.default_rng(seed)
    order = rng.permutation(E)
    logp = np.empty(E)
    logp[order] = -zipf_s * np.log(np.arange(1, E + 1))
    g = rng.gumbel(size=(T, E))
    return np.argsort(-(logp[None, :] + g), axis=1, kind="stable")[:, :k].astype(np.int32)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """uint16 view of a bf16 tensor's bits, on the host."""
    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def bits_to_bf16(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a, dtype=np.uint16)
    return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)


def load_stats(counts: np.ndarray) -> dict:
    """Summary of a per-expert histogram (for reporting)."""
    c = np.asarray(counts, dtype=np.float64)
    mean = c.mean() if c.size else 0.0
    srt = np.sort(c)[::-1]
    n = c.size
    gini = 0.0
    if c.sum() > 0:
        s = np.sort(c)
        gini = float((2 * np.arange(1, n + 1) - n - 1).dot(s) / (n * s.sum()))
    return {"max_over_mean": float(srt[0] / mean) if mean > 0 else 0.0,
            "n_empty": int((c == 0).sum()),
            "top8_share": float(srt[:8].sum() / c.sum()) if c.sum() > 0 else 0.0,
            "gini": gini}


if __name__ == "__main__":
    for name, wl in WORKLOADS.items():
        print(name, wl.describe(), "cap", wl.cap)
