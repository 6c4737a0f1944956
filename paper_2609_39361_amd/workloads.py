"""Seeded synthetic inputs for the LampAttention forward pass.

This module only draws random numbers and applies the input recipe (channel
scales, rotary position embedding, bf16 cast).  It holds none of the method's
arithmetic and is shared by the GPU path's tests and benchmark and by the
oracle's tests.

The five workloads are stand-ins for the paper's evaluation on real Qwen3 and
Gemma 3 activations (Sec. 4), whose weights and datasets are not available:
they have those models' attention shapes (heads, GQA groups, head dimension,
RoPE base, sliding window) and heavy-tailed channel statistics.

Recipe (fixed, so every run of every process draws the same tensors):
  * torch.Generator('cpu').manual_seed(seed); draws in fp32 in the order
    Q, K, V (then the per-config extras listed in `make_inputs`);
  * per-(head, channel) scales multiply Q (per query head) and K (per kv head);
    V is N(0,1) without scales;
  * RoPE (rotate-half pairs (c, c + d/2), inv_freq_i = base^(-2i/d), positions
    0..N-1, angles and cos/sin in fp64) is applied after the scales;
  * the result is cast to bf16 with round-to-nearest-even.
"""
from dataclasses import dataclass, field
import math

import numpy as np
import torch


@dataclass
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    N: int
    d: int
    causal: int
    window: int
    bq: int
    bk: int
    nk: int
    delta: float = 2.0 ** -8
    tau: float = 0.5
    seed: int = 0
    kind: str = "gauss"           # recipe family, see make_inputs
    rope_base: float = 0.0        # 0 = no rotary embedding
    scale_sigma: float = 0.0      # log-normal sigma of channel scales
    n_outlier: int = 0            # outlier channels (config 1/2 family)
    outlier_gain: float = 1.0
    sink_rows: int = 0            # key rows scaled by sink_gain per (b, h)
    sink_gain: float = 1.0
    M: int = 0                    # decode form: query rows per (b, h) at positions N-M .. N-1 (0: prefill)
    extra: dict = field(default_factory=dict)

    def replace(self, **kw):
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)

    @property
    def visible_logits(self):
        """Number of (query, key) pairs the mask leaves visible, all heads."""
        N, W = self.N, self.window
        if self.M > 0:   # query rows at positions N-M .. N-1 against N keys
            pos = np.arange(N - self.M, N)
            vis = np.full(self.M, N) if not self.causal else (pos + 1 if W <= 0 else np.minimum(pos + 1, W))
            return self.B * self.Hq * int(vis.sum())
        if not self.causal:
            per = N * N
        elif W <= 0 or W >= N:
            per = N * (N + 1) // 2
        else:
            per = W * (W + 1) // 2 + (N - W) * W
        return self.B * self.Hq * per

    @property
    def macs(self):
        """Emulated 8-bit multiply-adds: d per visible logit."""
        return self.visible_logits * self.d

    @property
    def eff_flops(self):
        """Effective attention FLOP: 4*B*H*N^2*d, halved for causal (decode
        form: 4*d per visible (query, key) pair)."""
        if self.M > 0:
            return 4.0 * self.d * self.visible_logits
        f = 4.0 * self.B * self.Hq * self.N * self.N * self.d
        return f / 2 if self.causal else f


# Block sizes (b_q, b_k, N_k): 64x64 and 128x64 "sub-blocks" for the first two
# configs, the paper's simulation tiling (128 queries x 64 keys in N_k = 4
# sub-blocks of 16 keys, Sec. 4.1) for the rest.
CONFIGS = {
    1: Workload("c1_single_head_n256_d64", 1, 1, 1, 256, 64, 0, 0, 64, 64, 4, seed=0,
                kind="outlier", n_outlier=2, outlier_gain=16.0),
    2: Workload("c2_mha8_n1024_d128_causal", 2, 8, 8, 1024, 128, 1, 0, 128, 64, 4, seed=1,
                kind="outlier", n_outlier=4, outlier_gain=12.0, sink_rows=10, sink_gain=8.0),
    3: Workload("c3_qwen3_8b_prefill_n8192", 1, 32, 8, 8192, 128, 1, 0, 128, 16, 4, seed=2,
                kind="rope_lognormal", rope_base=1e6, scale_sigma=0.75),
    4: Workload("c4_gemma3_4b_local_n16384_w1024", 1, 8, 4, 16384, 256, 1, 1024, 128, 16, 4, seed=3,
                kind="rope_lognormal", rope_base=1e4, scale_sigma=1.0),
    40: Workload("c4_gemma3_4b_global_n16384", 1, 8, 4, 16384, 256, 1, 0, 128, 16, 4, seed=3,
                 kind="rope_lognormal", rope_base=1e6, scale_sigma=1.0),
    5: Workload("c5_long_context_b4_n32768", 4, 32, 8, 32768, 128, 1, 0, 128, 16, 4, seed=4,
                kind="rope_student_t", rope_base=1e6),
    # Decode form (vector LAMP, Sec. 2, Eq. (6)): one new query row per
    # sequence against an 8K key/value cache, Qwen3-8B attention shape and
    # config-3 statistics; key tiles of 64 logits (bk), one row per update.
    6: Workload("c6_qwen3_8b_decode_b32_kv8192", 32, 32, 8, 8192, 128, 1, 0, 1, 64, 1, seed=5,
                kind="rope_lognormal", rope_base=1e6, scale_sigma=0.75, M=1),
}

TAU_SWEEP = [math.inf, 1.0, 0.5, 2.0 ** -5, 0.0]


def _rope_(x, base, pos0=0):
    """In-place rotate-half RoPE on x [..., N, d] (fp32); angles in fp64."""
    N, d = x.shape[-2], x.shape[-1]
    half = d // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    ang = np.arange(pos0, pos0 + N, dtype=np.float64)[:, None] * inv[None, :]
    c = torch.from_numpy(np.cos(ang).astype(np.float32))
    s = torch.from_numpy(np.sin(ang).astype(np.float32))
    x1 = x[..., :half].clone()
    x2 = x[..., half:].clone()
    x[..., :half] = x1 * c - x2 * s
    x[..., half:] = x2 * c + x1 * s
    return x


def make_inputs(w: Workload, device="cpu"):
    """(q, k, v) bf16 tensors [B,H,N,d] for workload `w`, drawn from its seed."""
    g = torch.Generator("cpu")
    g.manual_seed(int(w.seed))
    B, Hq, Hkv, N, d = w.B, w.Hq, w.Hkv, w.N, w.d
    nq = w.M if w.M > 0 else N          # decode form: the last M positions only
    q = torch.randn((B, Hq, nq, d), generator=g, dtype=torch.float32)
    k = torch.randn((B, Hkv, N, d), generator=g, dtype=torch.float32)
    v = torch.randn((B, Hkv, N, d), generator=g, dtype=torch.float32)
    if w.kind == "outlier":
        # A few outlier channels (the first n of a random permutation), scaled
        # on both Q and K; optionally "attention-sink-like" key rows: row 0
        # plus random others per (b, h), scaled by sink_gain.
        ch = torch.randperm(d, generator=g)[: w.n_outlier]
        q[..., ch] *= w.outlier_gain
        k[..., ch] *= w.outlier_gain
        if w.sink_rows > 0:
            for b in range(B):
                for h in range(Hkv):
                    others = torch.randperm(N - 1, generator=g)[: w.sink_rows - 1] + 1
                    rows = torch.cat([torch.zeros(1, dtype=torch.long), others])
                    k[b, h, rows, :] *= w.sink_gain
    elif w.kind in ("rope_lognormal", "rope_student_t"):
        if w.kind == "rope_lognormal":
            sq = torch.exp(w.scale_sigma * torch.randn((1, Hq, 1, d), generator=g))
            sk = torch.exp(w.scale_sigma * torch.randn((1, Hkv, 1, d), generator=g))
        else:
            # |T| with T ~ Student-t(3) = Z / sqrt(chi2_3 / 3).
            def student(shape):
                z = torch.randn(shape, generator=g)
                chi2 = (torch.randn(shape + (3,), generator=g) ** 2).sum(-1)
                return (z / torch.sqrt(chi2 / 3.0)).abs()
            sq = student((1, Hq, 1, d))
            sk = student((1, Hkv, 1, d))
        q *= sq
        k *= sk
        if w.rope_base > 0:
            _rope_(q, w.rope_base, N - nq)
            _rope_(k, w.rope_base)
    elif w.kind == "gauss":
        pass
    elif w.kind == "small_int":
        # Small integers: every partial sum is exactly representable in the
        # accumulator formats (used by tests).
        lim = int(w.extra.get("lim", 2))
        q = torch.randint(-lim, lim + 1, (B, Hq, nq, d), generator=g).float()
        k = torch.randint(-lim, lim + 1, (B, Hkv, N, d), generator=g).float()
        v = torch.randint(-lim, lim + 1, (B, Hkv, N, d), generator=g).float()
    else:
        raise ValueError("unknown workload kind %r" % w.kind)
    gain = float(w.extra.get("gain", 1.0))
    if gain != 1.0:
        q *= gain
        k *= gain
    # degenerate inputs for tests: all queries zero; every query and key row of
    # a head equal to its first row (all logits of a row equal)
    if w.extra.get("zero_q"):
        q.zero_()
    if w.extra.get("const"):
        q[:] = q[:, :, :1, :].clone()
        k[:] = k[:, :, :1, :].clone()
    if w.kind == "outlier" and w.M > 0:
        raise ValueError("outlier recipe is for the prefill form")
    out = tuple(t.to(torch.bfloat16).contiguous() for t in (q, k, v))
    if device != "cpu":
        out = tuple(t.to(device) for t in out)
    return out


def small(name="small", B=1, Hq=2, Hkv=1, N=128, d=64, causal=1, window=0, bq=64, bk=16, nk=4,
          seed=0, kind="rope_lognormal", **kw):
    """A small workload the oracle finishes in well under a second."""
    base = dict(rope_base=1e4, scale_sigma=0.75)
    base.update(kw)
    return Workload(name, B, Hq, Hkv, N, d, causal, window, bq, bk, nk, seed=seed, kind=kind, **base)
