"""Seeded synthetic inputs shared by the tests and the benchmark.

This module holds no 1.5-SPSA arithmetic: it only describes workload shapes and draws
seeded random inputs (weights, losses). The oracle and the GPU library both receive what
it produces; neither is imported here.

Shapes stand in for the models the paper trains (OPT-13B, OPT-30B; section 5, tables 1-2),
whose weights are not available: one flat parameter buffer laid out tensor by tensor in
OPT decoder order, matrices ~ N(0, 0.02), biases and LayerNorm beta 0, LayerNorm gamma 1.
Losses stand in for the forward passes (outside the sweep): i.i.d. N(2.0, 0.05).
"""

from dataclasses import dataclass

import numpy as np

OPT_VOCAB = 50272
OPT_POSITIONS = 2050  # 2048 positions plus the learned-embedding offset of 2


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str          # "f32" or "bf16"
    K: tuple            # probe counts per step that this workload is run with
    eps: float
    lr: float
    hidden: int = 0     # OPT shape; 0 for the flat tiny vector
    layers: int = 0
    ffn: int = 0
    n_flat: int = 0     # element count of the tiny flat vector

    @property
    def n(self):
        return self.n_flat if self.hidden == 0 else sum(sz for _, sz, _ in opt_tensors(self))


WORKLOADS = {
    "tiny": Workload("tiny", "f32", (4,), 1e-3, 1e-4, n_flat=1 << 20),
    "opt125m": Workload("opt125m", "bf16", (16,), 1e-3, 1e-3, 768, 12, 3072),
    "opt1.3b": Workload("opt1.3b", "bf16", (64,), 1e-3, 1e-3, 2048, 24, 8192),
    "opt13b": Workload("opt13b", "bf16", (16,), 1e-3, 1e-3, 5120, 40, 20480),
    "opt30b": Workload("opt30b", "bf16", (8, 32), 1e-3, 1e-3, 7168, 48, 28672),
}


def opt_tensors(w):
    """[(name, element count, init kind)] in buffer order; kind is 'normal', 'zero' or 'one'."""
    h, f = w.hidden, w.ffn
    out = [("embed_tokens", OPT_VOCAB * h, "normal"), ("embed_positions", OPT_POSITIONS * h, "normal")]
    for i in range(w.layers):
        p = f"layers.{i}."
        for proj in ("q_proj", "k_proj", "v_proj", "out_proj"):
            out += [(p + proj + ".weight", h * h, "normal"), (p + proj + ".bias", h, "zero")]
        out += [(p + "attn_ln.gamma", h, "one"), (p + "attn_ln.beta", h, "zero")]
        out += [(p + "fc1.weight", h * f, "normal"), (p + "fc1.bias", f, "zero")]
        out += [(p + "fc2.weight", f * h, "normal"), (p + "fc2.bias", h, "zero")]
        out += [(p + "final_ln.gamma", h, "one"), (p + "final_ln.beta", h, "zero")]
    out += [("final_ln.gamma", h, "one"), ("final_ln.beta", h, "zero")]
    return out


def tensor_offsets(w):
    """[(name, global offset, element count)] for the flat buffer."""
    res, o = [], 0
    for name, sz, _ in opt_tensors(w):
        res.append((name, o, sz))
        o += sz
    return res


def tiny_theta(n=1 << 20, seed=0):
    """The tiny fp32 vector: N(0, 0.02) from numpy's default generator, cast to float32."""
    return (np.random.default_rng(seed).standard_normal(n) * 0.02).astype(np.float32)


def synthetic_losses(K, seed):
    """(L_plus[K], L_minus[K], L_clean) ~ N(2.0, 0.05), drawn in that order."""
    rng = np.random.default_rng(seed)
    lp = rng.normal(2.0, 0.05, K)
    lm = rng.normal(2.0, 0.05, K)
    l0 = float(rng.normal(2.0, 0.05))
    return lp, lm, l0


def normal_f32(n, seed, scale=0.02):
    """Host float32 N(0, scale) values (for test windows and small buffers)."""
    return (np.random.default_rng(seed).standard_normal(n) * scale).astype(np.float32)


def normal_bf16_bits(n, seed, scale=0.02):
    """Host bf16 bit patterns of N(0, scale) values (round-to-nearest-even via torch)."""
    import torch
    x = torch.from_numpy(normal_f32(n, seed, scale))
    return x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def fill_opt_tensors_device(tensors, w):
    """Fill device tensors, one per OPT tensor in order (dtype matching w), with the OPT-shaped
    synthetic weights: each 'normal' tensor is drawn on the device from torch.Generator seeded
    1000 + index; biases and LayerNorm betas are 0 and gammas 1."""
    import torch
    for idx, ((name, sz, kind), t) in enumerate(zip(opt_tensors(w), tensors)):
        if t.numel() != sz:
            raise ValueError(f"tensor {idx} ({name}) holds {t.numel()} elements, expected {sz}")
        if kind == "zero":
            t.zero_()
        elif kind == "one":
            t.fill_(1.0)
        else:
            g = torch.Generator(device=t.device)
            g.manual_seed(1000 + idx)
            t.normal_(0.0, 0.02, generator=g)


def fill_opt_buffer_device(buf, w):
    """Fill a flat device tensor with the OPT-shaped synthetic weights, the tensors laid out back
    to back in order (the same values as fill_opt_tensors_device on separate tensors)."""
    views = [buf[o:o + sz] for _, o, sz in tensor_offsets(w)]
    fill_opt_tensors_device(views, w)


def stiff_paraboloid(d, kappa, seed):
    """The stiff paraboloid J(x) = x^T R^T diag(kappa, 1, ..., 1) R x with a random orthonormal
    R (section 5.3, appendix A.2), and a starting point x0 ~ N(0, 1) (float32).
    Returns (A = R^T diag R as float64 [d, d], x0)."""
    rng = np.random.default_rng(seed)
    R, _ = np.linalg.qr(rng.standard_normal((d, d)))
    A = R.T @ np.diag([float(kappa)] + [1.0] * (d - 1)) @ R
    x0 = rng.standard_normal(d).astype(np.float32)
    return A, x0
