"""Seeded synthetic inputs shared by the tests and the benchmark.

This module holds no 1.5-SPSA arithmetic: it only describes workload shapes and draws
seeded random inputs (weights, losses). The oracle and the GPU library both receive what
it produces; neither is imported here.

Shapes stand in for the models the paper trains (OPT-13B and OPT-30B, section 5 and
tables 1-2; Qwen3-8B and Qwen3-1.7B, section 5 "Qwen3 Post-Training"), whose weights are not
available: one parameter set laid out tensor by tensor in decoder order, matrices
~ N(0, 0.02), biases and LayerNorm beta 0, LayerNorm / RMSNorm gamma 1. Losses stand in for
the forward passes (outside the sweep): i.i.d. N(2.0, 0.05).
"""

from dataclasses import dataclass

import numpy as np

OPT_VOCAB = 50272
OPT_POSITIONS = 2050  # 2048 positions plus the learned-embedding offset of 2
QWEN3_VOCAB = 151936
QWEN3_HEAD_DIM = 128


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str          # "f32" or "bf16"
    K: tuple            # probe counts per step that this workload is run with
    eps: float
    lr: float
    hidden: int = 0     # model shape; 0 for the flat tiny vector
    layers: int = 0
    ffn: int = 0
    n_flat: int = 0     # element count of the tiny flat vector
    family: str = "opt"  # "opt" or "qwen3"
    heads: int = 0      # qwen3: query heads and key/value heads (head dimension 128)
    kv_heads: int = 0
    tied: bool = False  # qwen3: output projection shares the token embedding

    @property
    def n(self):
        return self.n_flat if self.hidden == 0 else sum(sz for _, sz, _ in model_tensors(self))


WORKLOADS = {
    "tiny": Workload("tiny", "f32", (4,), 1e-3, 1e-4, n_flat=1 << 20),
    "opt125m": Workload("opt125m", "bf16", (16,), 1e-3, 1e-3, 768, 12, 3072),
    "opt1.3b": Workload("opt1.3b", "bf16", (64,), 1e-3, 1e-3, 2048, 24, 8192),
    "opt13b": Workload("opt13b", "bf16", (16,), 1e-3, 1e-3, 5120, 40, 20480),
    "opt30b": Workload("opt30b", "bf16", (8, 32), 1e-3, 1e-3, 7168, 48, 28672),
    # the paper's Qwen3 runs use 60 probes per step and lr = eps = 1e-4 (appendix,
    # experiment configurations)
    "qwen3-1.7b": Workload("qwen3-1.7b", "bf16", (60,), 1e-4, 1e-4, 2048, 28, 6144, family="qwen3",
                           heads=16, kv_heads=8, tied=True),
    "qwen3-8b": Workload("qwen3-8b", "bf16", (60,), 1e-4, 1e-4, 4096, 36, 12288, family="qwen3",
                         heads=32, kv_heads=8, tied=False),
}


def opt_tensors(w):
    """OPT decoder: [(name, element count, init kind)] in buffer order; kind is 'normal',
    'zero' or 'one'."""
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


def qwen3_tensors(w):
    """Qwen3 decoder (grouped-query attention with per-head RMSNorm on queries and keys,
    SwiGLU MLP, no biases): [(name, element count, init kind)] in buffer order."""
    h, f, d = w.hidden, w.ffn, QWEN3_HEAD_DIM
    q, kv = w.heads * d, w.kv_heads * d
    out = [("embed_tokens", QWEN3_VOCAB * h, "normal")]
    for i in range(w.layers):
        p = f"layers.{i}."
        out += [(p + "input_norm.gamma", h, "one"),
                (p + "q_proj.weight", q * h, "normal"), (p + "k_proj.weight", kv * h, "normal"),
                (p + "v_proj.weight", kv * h, "normal"), (p + "o_proj.weight", h * q, "normal"),
                (p + "q_norm.gamma", d, "one"), (p + "k_norm.gamma", d, "one"),
                (p + "post_attn_norm.gamma", h, "one"),
                (p + "gate_proj.weight", f * h, "normal"), (p + "up_proj.weight", f * h, "normal"),
                (p + "down_proj.weight", h * f, "normal")]
    out += [("final_norm.gamma", h, "one")]
    if not w.tied:
        out += [("lm_head.weight", QWEN3_VOCAB * h, "normal")]
    return out


def model_tensors(w):
    """[(name, element count, init kind)] of a model-shaped workload, in buffer order."""
    return qwen3_tensors(w) if w.family == "qwen3" else opt_tensors(w)


def tensor_offsets(w):
    """[(name, global offset, element count)] for the flat buffer."""
    res, o = [], 0
    for name, sz, _ in model_tensors(w):
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


def fill_model_tensors_device(tensors, w):
    """Fill device tensors, one per model tensor in order (dtype matching w), with the
    model-shaped synthetic weights: each 'normal' tensor is drawn on the device from torch.Generator seeded
    1000 + index; biases and norm betas are 0 and gammas 1."""
    import torch
    for idx, ((name, sz, kind), t) in enumerate(zip(model_tensors(w), tensors)):
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


def fill_model_buffer_device(buf, w):
    """Fill a flat device tensor with the model-shaped synthetic weights, the tensors laid out
    back to back in order (the same values as fill_model_tensors_device on separate tensors)."""
    views = [buf[o:o + sz] for _, o, sz in tensor_offsets(w)]
    fill_model_tensors_device(views, w)


def stiff_paraboloid(d, kappa, seed):
    """The stiff paraboloid J(x) = x^T R^T diag(kappa, 1, ..., 1) R x with a random orthonormal
    R (section 5.3, appendix A.2), and a starting point x0 ~ N(0, 1) (float32).
    Returns (A = R^T diag R as float64 [d, d], x0)."""
    rng = np.random.default_rng(seed)
    R, _ = np.linalg.qr(rng.standard_normal((d, d)))
    A = R.T @ np.diag([float(kappa)] + [1.0] * (d - 1)) @ R
    x0 = rng.standard_normal(d).astype(np.float32)
    return A, x0
