"""Seeded synthetic inputs shaped like the paper's calibration workload.

The paper calibrates on 1248 WikiText2 sequences of 2048 tokens with a global batch of 32
(Sec. 4.1); neither the dataset nor the model weights are available here, so every tensor is drawn
from a seeded generator with the shapes of the decoder blocks being calibrated. Each tensor gets its
own generator stream keyed by (workload, tensor name, seed). The same bytes feed the HIP path and
the CPU oracle. This module holds none of the method's arithmetic: it only draws numbers.

Recipes:
  * weights: N(0, sigma^2); then exactly round(p * N * K) distinct, uniformly chosen entries are
    multiplied by a factor f (sparse outliers).
  * activations: i.i.d. N(0, 1) per element, or Student-t with 3 degrees of freedom
    (Z / sqrt(chi2_3 / 3)); then exactly round(p * K) distinct input channels (whole columns) are
    multiplied by f. A fresh channel set per input tensor.
  * the reference output of a layer is the unquantised product X W^T (fp32 accumulation), stored
    in the operand dtype.
  * a perturbed parameter state multiplies each learnable scale by 2^U[-0.5, 0.5] and draws each
    coefficient from U[0.75, 1.25].
"""
from __future__ import annotations

import zlib
from dataclasses import dataclass, field

import torch

MXFP4 = 0
NVFP4 = 1


@dataclass(frozen=True)
class Linear:
    name: str
    N: int          # output features
    K: int          # input features (the block / reduction dimension)
    source: str     # name of the activation tensor that feeds it


@dataclass(frozen=True)
class Workload:
    name: str
    fmt: int
    sub_block: int
    M: int                          # calibration tokens in one step
    linears: tuple
    inputs: dict = field(hash=False)  # activation name -> K
    dtype: str = "bf16"             # operand dtype: "bf16" or "f32"
    w_sigma: float = 0.02
    w_outlier_p: float = 0.001
    w_outlier_f: float = 10.0
    x_kind: str = "normal"          # "normal", "student_t3" or "lowrank"
    x_outlier_p: float = 0.01
    x_outlier_f: float = 30.0
    seed: int = 0

    @property
    def block(self) -> int:
        return 32 if self.fmt == MXFP4 else 16


def decoder_block_linears(hidden: int, q_heads: int, kv_heads: int, head_dim: int, mlp: int):
    """The seven linears of a decoder block and the four distinct activations feeding them."""
    q, kv = q_heads * head_dim, kv_heads * head_dim
    linears = (
        Linear("q_proj", q, hidden, "attn_in"),
        Linear("k_proj", kv, hidden, "attn_in"),
        Linear("v_proj", kv, hidden, "attn_in"),
        Linear("o_proj", hidden, q, "o_in"),
        Linear("gate_proj", mlp, hidden, "mlp_in"),
        Linear("up_proj", mlp, hidden, "mlp_in"),
        Linear("down_proj", hidden, mlp, "down_in"),
    )
    inputs = {"attn_in": hidden, "o_in": q, "mlp_in": hidden, "down_in": mlp}
    return linears, inputs


def _block(name, fmt, M, hidden, q_heads, kv_heads, mlp, **kw) -> Workload:
    linears, inputs = decoder_block_linears(hidden, q_heads, kv_heads, 128, mlp)
    return Workload(name=name, fmt=fmt, sub_block=8, M=M, linears=linears, inputs=inputs, **kw)


WORKLOADS = {
    # one 256x256 fp32 linear, 128 tokens, MXFP4 with one coefficient per sub-block of 8
    "linear256_mxfp4_f32": Workload(
        name="linear256_mxfp4_f32", fmt=MXFP4, sub_block=8, M=128,
        linears=(Linear("linear", 256, 256, "x"),), inputs={"x": 256}, dtype="f32",
        w_sigma=0.02, w_outlier_p=0.001, w_outlier_f=10.0,
        x_kind="normal", x_outlier_p=4 / 256, x_outlier_f=20.0),
    # hidden 2560, 32 q / 8 kv heads of 128, MLP 9728, 32 x 2048 tokens, MXFP4
    "block2560_mxfp4": _block("block2560_mxfp4", MXFP4, 65536, 2560, 32, 8, 9728,
                              w_sigma=0.02, w_outlier_p=0.001, w_outlier_f=10.0,
                              x_kind="normal", x_outlier_p=0.01, x_outlier_f=30.0),
    # the same shapes under NVFP4 with heavy-tailed Student-t(3) activations
    "block2560_nvfp4": _block("block2560_nvfp4", NVFP4, 65536, 2560, 32, 8, 9728,
                              w_sigma=0.02, w_outlier_p=0.001, w_outlier_f=10.0,
                              x_kind="student_t3", x_outlier_p=0.0, x_outlier_f=1.0),
    # hidden 4096, 32 q / 8 kv heads, MLP 14336, 128 x 2048 tokens, MXFP4
    "block4096_mxfp4": _block("block4096_mxfp4", MXFP4, 262144, 4096, 32, 8, 14336,
                              w_sigma=0.015, w_outlier_p=0.0005, w_outlier_f=15.0,
                              x_kind="normal", x_outlier_p=0.005, x_outlier_f=50.0),
    # hidden 8192, 64 q / 8 kv heads, MLP 28672, 64 x 2048 tokens, MXFP4, plus export
    "block8192_mxfp4": _block("block8192_mxfp4", MXFP4, 131072, 8192, 64, 8, 28672,
                              w_sigma=0.01, w_outlier_p=0.001, w_outlier_f=10.0,
                              x_kind="normal", x_outlier_p=0.01, x_outlier_f=30.0),
}


def scaled(w: Workload, M: int | None = None, hidden_div: int = 1, name: str | None = None) -> Workload:
    """A smaller copy of a workload (fewer tokens and/or narrower layers) with the same recipe."""
    linears = tuple(Linear(l.name, max(l.N // hidden_div, 1), l.K // hidden_div, l.source)
                    for l in w.linears)
    inputs = {k: v // hidden_div for k, v in w.inputs.items()}
    return Workload(name=name or f"{w.name}_small", fmt=w.fmt, sub_block=w.sub_block,
                    M=M or w.M, linears=linears, inputs=inputs, dtype=w.dtype, w_sigma=w.w_sigma,
                    w_outlier_p=w.w_outlier_p, w_outlier_f=w.w_outlier_f, x_kind=w.x_kind,
                    x_outlier_p=w.x_outlier_p, x_outlier_f=w.x_outlier_f, seed=w.seed)


def _generator(workload: str, tensor: str, seed: int, device) -> torch.Generator:
    key = zlib.crc32(f"{workload}/{tensor}".encode()) ^ (seed * 0x9E3779B1 & 0xFFFFFFFF)
    g = torch.Generator(device=device)
    g.manual_seed(key)
    return g


def _torch_dtype(name: str):
    return torch.bfloat16 if name == "bf16" else torch.float32


def weight(w: Workload, linear: Linear, device="cpu", outlier_rows: list | None = None) -> torch.Tensor:
    """W [N][K]: N(0, sigma^2) with round(p N K) entries multiplied by f.

    If ``outlier_rows`` is a list, the sorted distinct rows holding an outlier are appended to it.
    """
    g = _generator(w.name, linear.name + ".weight", w.seed, device)
    W = torch.randn(linear.N, linear.K, generator=g, device=device, dtype=torch.float32) * w.w_sigma
    count = int(round(w.w_outlier_p * linear.N * linear.K))
    if count:
        idx = torch.randperm(linear.N * linear.K, generator=g, device=device)[:count]
        W.view(-1)[idx] *= w.w_outlier_f
        if outlier_rows is not None:
            outlier_rows.extend(sorted(set((idx // linear.K).cpu().tolist())))
    return W.to(_torch_dtype(w.dtype)).contiguous()


def activation(w: Workload, source: str, M: int | None = None, device="cpu") -> torch.Tensor:
    """X [M][K] for one activation tensor of the block."""
    K = w.inputs[source]
    M = M or w.M
    g = _generator(w.name, source + ".act", w.seed, device)
    if w.x_kind == "student_t3":
        z = torch.randn(M, K, generator=g, device=device)
        chi2 = torch.zeros(M, K, device=device)
        for _ in range(3):
            chi2 += torch.randn(M, K, generator=g, device=device) ** 2
        X = z / torch.sqrt(chi2 / 3.0)
    else:
        X = torch.randn(M, K, generator=g, device=device)
    count = int(round(w.x_outlier_p * K))
    if count:
        ch = torch.randperm(K, generator=g, device=device)[:count]
        X[:, ch] *= w.x_outlier_f
    return X.to(_torch_dtype(w.dtype)).contiguous()


LOWRANK_RANK = 32
LOWRANK_NOISE = 0.1


def _lowrank(w: Workload, source: str, M: int, K: int, g: torch.Generator, device) -> torch.Tensor:
    """Correlated channels: X = Z A + 0.1 E with a fixed mixing matrix A [32][K] (entries N(0, 1/32),
    drawn once per input tensor), fresh latent factors Z [M][32] and noise E, both N(0, 1). Every
    channel has about unit variance and the channels are strongly correlated, so X^T X is far from
    diagonal, as in the inputs of real decoder layers."""
    A = torch.randn(LOWRANK_RANK, K, generator=_generator(w.name, source + ".mixing", w.seed, device),
                    device=device) / LOWRANK_RANK ** 0.5
    Z = torch.randn(M, LOWRANK_RANK, generator=g, device=device)
    return Z @ A + LOWRANK_NOISE * torch.randn(M, K, generator=g, device=device)


def activation_batch(w: Workload, source: str, step: int, M: int | None = None, device="cpu") -> torch.Tensor:
    """Batch `step` of a calibration epoch for one activation tensor of the block: fresh tokens from
    a stream keyed by the step, the same outlier channels (same scale factor) in every batch, as
    tokens of one layer input drawn from a fixed distribution."""
    K = w.inputs[source]
    M = M or w.M
    g = _generator(w.name, f"{source}.act.batch{step}", w.seed, device)
    if w.x_kind == "lowrank":
        X = _lowrank(w, source, M, K, g, device)
    elif w.x_kind == "student_t3":
        z = torch.randn(M, K, generator=g, device=device)
        chi2 = torch.zeros(M, K, device=device)
        for _ in range(3):
            chi2 += torch.randn(M, K, generator=g, device=device) ** 2
        X = z / torch.sqrt(chi2 / 3.0)
    else:
        X = torch.randn(M, K, generator=g, device=device)
    count = int(round(w.x_outlier_p * K))
    if count:
        ch = torch.randperm(K, generator=_generator(w.name, source + ".channels", w.seed, device), device=device)
        X[:, ch[:count]] *= w.x_outlier_f
    return X.to(_torch_dtype(w.dtype)).contiguous()


def reference_output(X: torch.Tensor, W: torch.Tensor) -> torch.Tensor:
    """Y_ref = X W^T of the unquantised layer with fp32 accumulation, in X's dtype."""
    if X.dtype == torch.float32 or X.device.type == "cpu":
        Y = torch.mm(X.float(), W.float().t().contiguous())
    else:
        Y = torch.mm(X, W.t().contiguous())
    return Y.to(X.dtype).contiguous()


def perturb(s_fp: torch.Tensor, c: torch.Tensor, w: Workload, tag: str):
    """A seeded non-initial parameter state: s_fp * 2^U[-0.5,0.5], c ~ U[0.75, 1.25]."""
    g = _generator(w.name, tag + ".perturb", w.seed, s_fp.device)
    e = torch.rand(s_fp.shape, generator=g, device=s_fp.device) - 0.5
    s_new = (s_fp.float() * torch.exp2(e)).contiguous()
    c_new = (0.75 + 0.5 * torch.rand(c.shape, generator=g, device=c.device)).contiguous()
    return s_new, c_new
