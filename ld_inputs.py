"""Seeded synthetic inputs for the layer-dropout hot path.

This module only draws random tensors; it holds none of the method's
arithmetic.  Both the HIP path (through its tests and the benchmark) and the
CPU oracle are fed from it, so both see exactly the same values.

Recipe (all configurations are synthetic; the paper's corpus is not used):
  * each tensor comes from numpy.random.default_rng(SeedSequence([seed,
    tensor_id, layer])) as float32 standard normals times a scale;
  * hidden states X^0 ~ N(0, 1); weight matrices ~ N(0, 0.02);
    RMSNorm gains = 1 (or 1 + N(0, 0.02) with gain_jitter, which exposes
    gain-indexing mistakes); upstream gradient dL/dX^L ~ N(0, 1);
  * for bf16 configurations the float32 draws are rounded to bfloat16
    (round to nearest even, by torch's conversion) and the oracle consumes the
    same bf16 values widened to float64, so a comparison measures kernel error
    and not input quantisation.
Tensor ids: x 0, g_attn 1, w_qkv 2, w_o 3, g_mlp 4, w_gate_up 5, w_down 6,
upstream gradient 7.
"""

from dataclasses import dataclass

import numpy as np
import torch

TENSOR_IDS = dict(x=0, g_attn=1, w_qkv=2, w_o=3, g_mlp=4, w_gate_up=5, w_down=6, gy=7)
WEIGHT_KEYS = ("g_attn", "w_qkv", "w_o", "g_mlp", "w_gate_up", "w_down")


@dataclass(frozen=True)
class Shape:
    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int
    seq: int
    batch: int
    dtype: str  # "f32" or "bf16"
    kind: int = 0  # block kind: 0 SwiGLU, 1 ALiBi + squared ReLU (W_up only)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


# The workloads of the hot path (names say what they are).
SHAPES = {
    "tiny": Shape(2, 64, 4, 172, 32, 8, "f32"),
    "125m": Shape(12, 768, 12, 2048, 1024, 8, "bf16"),
    "1b": Shape(16, 2048, 16, 5504, 2048, 8, "bf16"),
    "7b": Shape(32, 4096, 32, 11008, 4096, 4, "bf16"),
    "1b_b32": Shape(16, 2048, 16, 5504, 2048, 32, "bf16"),
    # the paper's 3.9B architecture (architecture table: d 2048, 40 layers,
    # 16 heads of 128, FFN multiplier 8) with its block (ALiBi, squared ReLU);
    # sequence length and batch as the 1B workload (the paper states neither)
    "paper_3p9b": Shape(40, 2048, 16, 16384, 2048, 8, "bf16", 1),
}


def _normal(shape, seed, tensor_id, layer, scale):
    rng = np.random.default_rng(np.random.SeedSequence([seed, tensor_id, layer]))
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(scale)


def _cast(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype)


def weight_shapes(sh):
    d, f = sh.d_model, sh.d_ff
    return dict(g_attn=(d,), w_qkv=(3 * d, d), w_o=(d, d), g_mlp=(d,),
                w_gate_up=((2 if sh.kind == 0 else 1) * f, d), w_down=(d, f))


def layer_weights(sh, layer, seed=0, gain_jitter=False):
    """Dict of CPU tensors in the configuration's dtype for one layer."""
    out = {}
    for k, shp in weight_shapes(sh).items():
        if k in ("g_attn", "g_mlp"):
            a = np.ones(shp, dtype=np.float32)
            if gain_jitter:
                a = a + _normal(shp, seed, TENSOR_IDS[k], layer, 0.02)
        else:
            a = _normal(shp, seed, TENSOR_IDS[k], layer, 0.02)
        out[k] = _cast(a, sh.torch_dtype)
    return out


def hidden(sh, seed=0, batch=None):
    b = sh.batch if batch is None else batch
    return _cast(_normal((b, sh.seq, sh.d_model), seed, TENSOR_IDS["x"], 0, 1.0), sh.torch_dtype)


def upstream_grad(sh, seed=0, batch=None):
    b = sh.batch if batch is None else batch
    return _cast(_normal((b, sh.seq, sh.d_model), seed, TENSOR_IDS["gy"], 0, 1.0), sh.torch_dtype)


def f64(t):
    """The exact values of a CPU tensor as a float64 numpy array."""
    return t.detach().to(torch.float64).numpy()


def _device_seed(seed, tensor_id, layer):
    return (seed * 1_000_003 + tensor_id * 10_007 + layer) & 0x7FFFFFFFFFFFFFFF


def _device_normal(shape, seed, tensor_id, layer, scale, dtype, device):
    g = torch.Generator(device=device)
    g.manual_seed(_device_seed(seed, tensor_id, layer))
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    return (t * scale).to(dtype)


def device_layer_weights(sh, layer, device, seed=0):
    """Same distributions as layer_weights, drawn on the device with torch's
    seeded generator (used where numpy would take minutes: the benchmark)."""
    out = {}
    for k, shp in weight_shapes(sh).items():
        if k in ("g_attn", "g_mlp"):
            out[k] = torch.ones(shp, dtype=sh.torch_dtype, device=device)
        else:
            out[k] = _device_normal(shp, seed, TENSOR_IDS[k], layer, 0.02, sh.torch_dtype, device)
    return out


def device_hidden(sh, device, seed=0):
    return _device_normal((sh.batch, sh.seq, sh.d_model), seed, TENSOR_IDS["x"], 0, 1.0,
                          sh.torch_dtype, device)


def device_upstream_grad(sh, device, seed=0):
    return _device_normal((sh.batch, sh.seq, sh.d_model), seed, TENSOR_IDS["gy"], 0, 1.0,
                          sh.torch_dtype, device)
