"""Seeded synthetic inputs for the DF-SSM scaffold + int8 LoRA linear.

This module only draws random numbers in the layouts the library takes; it
holds none of the method's arithmetic and imports neither the oracle nor the
GPU package, so both sides can be fed the same bytes.

Shapes follow Mamba-2 (the paper's model, Sec. 3 / Table 1): the 1.3B model
has d_model 2048 and 48 layers, in_proj 2048 -> 8512 (2*4096 + 2*128 + 64)
and out_proj 4096 -> 2048; the 130M model has d_model 768 and in_proj
768 -> 3352.  No trained weights are available, so every tensor is drawn:

  sign bits   i.i.d. Bernoulli(1/2), packed 32 per uint32, [N][K/32]
  alpha       U(0.01, 0.05) fp32 per output row
  A, B        int8 uniform on [-127, 127]   (A: [r,K], B: [N,r])
  beta        U(1e-4, 1e-3) fp32 per output row (times beta_scale)
  x           fp16 N(0,1), with a fixed seeded set of round(0.01*K) input
              channels multiplied by 20 (activation outliers)
  E           int8 embedding table [V, d]: round(N(0,1) * 32) clipped to
              [-127, 127] (a Gaussian row quantised with absmax near 4 sigma)
  scale       U(2e-4, 1e-3) fp32 per table row
  tok         int32 token ids, uniform on [0, V)

The tied embedding of the 1.3B model is 50,280 x 2048 (Table 1: 103 MB in
int8).

Mamba-2 decode-step parameters and state (d_inner = 2 d_model, heads of 64
channels, d_state 128 for the 1.3B model, one B/C group, d_conv 4):

  conv_w      U(-0.5, 0.5) fp32 [conv_dim][4];  conv_b U(-0.1, 0.1)
  dt_bias     U(-6.9, -2.3) (softplus of it spans about 1e-3 .. 0.1)
  A_log       U(0, 2.77)    (A = -exp(A_log) spans -1 .. -16)
  D           U(0.5, 1.5);  norm weights U(0.8, 1.2)
  conv state  N(0, 1) [M][conv_dim][4];  SSM state 0.5 N(0, 1) [M][H][P][N]
  in_proj out N(0, 1) fp32 [M][2 d_inner + 2 N + H];  residual N(0, 1)

Each tensor set has its own numpy PCG64 stream keyed by
(config, layer, projection, variant), so sets never share a stream.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Tuple

import numpy as np

# 1.3B Mamba-2 projection shapes (K = input features, N = output features)
IN_PROJ_1P3B = (2048, 8512)
OUT_PROJ_1P3B = (4096, 2048)
N_LAYERS_1P3B = 48
VOCAB_1P3B = 50280
D_MODEL_1P3B = 2048


@dataclass(frozen=True)
class Config:
    name: str
    M: Tuple[int, ...]
    K: int
    N: int
    r: int
    doc: str


CONFIGS: Dict[int, Config] = {
    0: Config("130m_in_proj_m1", (1,), 768, 3352, 16, "Mamba-2-130M in_proj, one token"),
    1: Config("1p3b_in_proj_m1", (1,), 2048, 8512, 64, "Mamba-2-1.3B in_proj decode, one token"),
    2: Config("1p3b_out_proj_small_m", (1, 4, 8, 16, 32), 4096, 2048, 64,
              "Mamba-2-1.3B out_proj, small-batch decode"),
    3: Config("1p3b_decode_sweep", (1,), 0, 0, 64,
              "48 x (in_proj 2048->8512, out_proj 4096->2048), each output re-quantised"),
    4: Config("1p3b_in_proj_prefill", (2048,), 2048, 8512, 64, "Mamba-2-1.3B in_proj, 2048-token prefill"),
}


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng([int(k) for k in key])


def weights(K: int, N: int, r: int, key=(0, 0, 0, 0), beta_scale: float = 1.0) -> dict:
    """One weight set: packed sign bits, alpha, A, B, beta (numpy, host)."""
    if K % 32:
        raise ValueError("K must be a multiple of 32")
    g = _rng(1, *key)
    bits = g.integers(0, 2 ** 32, size=(N, K // 32), dtype=np.uint32)
    alpha = g.uniform(0.01, 0.05, size=N).astype(np.float32)
    A = g.integers(-127, 128, size=(r, K), dtype=np.int8)
    B = g.integers(-127, 128, size=(N, r), dtype=np.int8)
    beta = (g.uniform(1e-4, 1e-3, size=N) * beta_scale).astype(np.float32)
    return dict(w_bits=bits, alpha=alpha, A=A, B=B, beta=beta)


def activations(M: int, K: int, key=(0, 0), dtype=np.float16, outlier_frac: float = 0.01,
                outlier_gain: float = 20.0) -> np.ndarray:
    """x [M,K]: N(0,1) with a fixed set of outlier channels scaled by outlier_gain."""
    g = _rng(2, *key)
    z = g.standard_normal((M, K), dtype=np.float32)
    n_out = int(round(outlier_frac * K))
    if n_out:
        ch = g.choice(K, n_out, replace=False)
        z[:, ch] *= np.float32(outlier_gain)
    return z.astype(dtype)


def config_weights(cfg: int, variant: int = 0, beta_scale: float = 1.0) -> dict:
    c = CONFIGS[cfg]
    return weights(c.K, c.N, c.r, key=(cfg, 0, 0, variant), beta_scale=beta_scale)


def config_activations(cfg: int, M: int, variant: int = 0) -> np.ndarray:
    c = CONFIGS[cfg]
    return activations(M, c.K, key=(cfg, 999_999 + variant))


def sweep_shapes(n_layers: int = N_LAYERS_1P3B) -> List[Tuple[int, int]]:
    """(K, N) of every linear of the decode sweep: in_proj, out_proj, ... ."""
    out = []
    for _ in range(n_layers):
        out.append(IN_PROJ_1P3B)
        out.append(OUT_PROJ_1P3B)
    return out


def sweep_weights(n_layers: int = N_LAYERS_1P3B, r: int = 64, variant: int = 0,
                  beta_scale: float = 1.0, shapes=None) -> List[dict]:
    """The decode sweep's weight sets, one per linear (2 per layer)."""
    shapes = sweep_shapes(n_layers) if shapes is None else shapes
    out = []
    for i, (K, N) in enumerate(shapes):
        out.append(weights(K, N, r, key=(3, i // 2, i % 2, variant), beta_scale=beta_scale))
    return out


def sweep_input(M: int = 1, K: int = IN_PROJ_1P3B[0], variant: int = 0) -> np.ndarray:
    return activations(M, K, key=(3, 999_999 + variant))


def weight_bytes(ws: dict) -> int:
    """Bytes of one weight set as stored: signs + A + B + alpha + beta."""
    return int(sum(ws[k].nbytes for k in ("w_bits", "A", "B", "alpha", "beta")))


def embedding(V: int, d: int, key=(0,)) -> Tuple[np.ndarray, np.ndarray]:
    """(E int8 [V, d], scale fp32 [V]) of a tied int8 embedding table."""
    g = _rng(4, *key)
    z = g.standard_normal((V, d), dtype=np.float32)
    z *= np.float32(32.0)
    np.rint(z, out=z)
    np.clip(z, -127, 127, out=z)
    scale = g.uniform(2e-4, 1e-3, size=V).astype(np.float32)
    return z.astype(np.int8), scale


def tokens(M: int, V: int, key=(0,)) -> np.ndarray:
    """int32 token ids [M], uniform on [0, V)."""
    return _rng(5, *key).integers(0, V, size=M, dtype=np.int32)


def mamba_dims(d_model: int, d_state: int = 128, headdim: int = 64) -> dict:
    """Sizes of one Mamba-2 mixer (one B/C group, d_conv 4)."""
    d_inner = 2 * d_model
    H = d_inner // headdim
    conv_dim = d_inner + 2 * d_state
    return dict(d_model=d_model, d_inner=d_inner, d_state=d_state, headdim=headdim, nheads=H,
                conv_dim=conv_dim, ld=d_inner + conv_dim + H)


def mamba_params(d_model: int, d_state: int = 128, headdim: int = 64, key=(0,)) -> dict:
    """Per-layer parameters of the step around the linears (numpy, host)."""
    dm = mamba_dims(d_model, d_state, headdim)
    g = _rng(6, *key)
    f = np.float32
    return dict(conv_w=g.uniform(-0.5, 0.5, (dm["conv_dim"], 4)).astype(f),
                conv_b=g.uniform(-0.1, 0.1, dm["conv_dim"]).astype(f),
                dt_bias=g.uniform(-6.9, -2.3, dm["nheads"]).astype(f),
                A_log=g.uniform(0.0, 2.77, dm["nheads"]).astype(f),
                D=g.uniform(0.5, 1.5, dm["nheads"]).astype(f),
                norm_w=g.uniform(0.8, 1.2, d_model).astype(f),
                gate_w=g.uniform(0.8, 1.2, dm["d_inner"]).astype(f))


def mamba_state(M: int, d_model: int, d_state: int = 128, headdim: int = 64, key=(0,)) -> dict:
    """conv_state [M][conv_dim][4] (position 3 newest) and ssm_state [M][H][P][N]."""
    dm = mamba_dims(d_model, d_state, headdim)
    g = _rng(7, *key)
    conv = g.standard_normal((M, dm["conv_dim"], 4), dtype=np.float32)
    ssm = g.standard_normal((M, dm["nheads"], headdim, d_state), dtype=np.float32)
    ssm *= np.float32(0.5)
    return dict(conv_state=conv, ssm_state=ssm)


def inproj_out(M: int, d_model: int, d_state: int = 128, headdim: int = 64, key=(0,)) -> np.ndarray:
    """A stand-in for in_proj's fp32 output rows [z | x | B | C | dt]."""
    dm = mamba_dims(d_model, d_state, headdim)
    return _rng(8, *key).standard_normal((M, dm["ld"]), dtype=np.float32)


def residual(M: int, d_model: int, key=(0,)) -> np.ndarray:
    return _rng(9, *key).standard_normal((M, d_model), dtype=np.float32)


def weights_i4(K: int, N: int, r: int, key=(0, 0, 0, 0), beta_scale: float = 1.0) -> dict:
    """A weight set with int4 LoRA factors: the int8 set's signs and scales,
    A4 [r][K/2] and B4 [N][r/2] as uniform random bytes (every nibble value
    -8..7 equally likely, two per byte).  r must be even."""
    if r % 2:
        raise ValueError("r must be even for packed int4 factors")
    ws = weights(K, N, 0, key=key)
    g = _rng(10, *key)
    A4 = g.integers(0, 256, size=(r, K // 2), dtype=np.uint8)
    B4 = g.integers(0, 256, size=(N, r // 2), dtype=np.uint8)
    beta = (g.uniform(1e-4, 1e-3, size=N) * beta_scale).astype(np.float32)
    return dict(w_bits=ws["w_bits"], alpha=ws["alpha"], A4=A4, B4=B4, beta=beta)
