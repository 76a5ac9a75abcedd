"""Seeded synthetic weight tensors shaped like the paper's evaluated models.

This module only *draws inputs*. It contains none of the codec's arithmetic
(no field split, histogram, normalisation or rANS step), so both the CPU
oracle and the HIP decode path can be fed from it without sharing any of the
method.

The paper measures real checkpoints (Qwen, Mistral, DeepSeek, Mixtral, Llama;
Sec. VI-A); those weights are not available here, so seeded draws with the
same tensor shapes, storage formats and value statistics stand in for them:

* bf16 weights: i.i.d. Normal(0, sigma) in PyTorch ``[out, in]`` layout,
  optionally with 0.1 % of the *input* columns scaled by 20 (outlier
  channels), rounded to bf16 with round-to-nearest-even;
* RMSNorm vectors: Normal(1, 0.02) rounded to bf16;
* int4: symmetric per-group quantisation (group 128 along the input dim),
  fp16 scale = absmax/7, codes clamp(rint(w/scale), -8, 7) stored as two's
  complement nibbles, two per byte, low nibble = even element;
* int8 (SmoothQuant-style weights): per-output-row fp16 scale = absmax/127,
  codes clamp(rint(w/scale), -127, 127), weights 0.02 * Student-t(nu=5).

Every array is returned as the raw little-endian storage of the tensor:
``uint16`` for bf16/fp16, ``uint8`` for int8 codes and packed int4 bytes.

Two generation backends exist.  ``numpy`` (PCG64 streams keyed by
``SeedSequence``; the reference recipe used by every test) is generated in
row blocks on a thread pool, each block with its own child stream, so the
values do not depend on the thread count.  ``torch`` draws the 70B-layer
tensors on the GPU (for the sustained multi-layer benchmark, where host-side
drawing of ~68 G values would dominate the run); it follows the same recipe
with torch's device generator, so its values differ from the numpy draw of
the same seed.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

# Rows per generation block are chosen so a block holds about this many values.
_BLOCK_VALUES = 1 << 21


@dataclass
class Tensor:
    name: str
    dtype: str          # 'bf16' | 'fp16' | 'u8' | 'u4'
    data: np.ndarray    # raw storage (uint16 for 16-bit types, uint8 otherwise)
    shape: tuple        # logical shape in elements

    @property
    def nbytes(self) -> int:
        return int(self.data.nbytes)


def _threads() -> int:
    env = os.environ.get("WC_SYNTH_THREADS")
    if env:
        return max(1, int(env))
    return max(1, min(16, os.cpu_count() or 1))


def _pool_map(fn, items):
    items = list(items)
    if len(items) <= 1:
        return [fn(i) for i in items]
    with ThreadPoolExecutor(_threads()) as ex:
        return list(ex.map(fn, items))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); finite inputs only."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) >> 16).astype(np.uint16)


def _key(*parts) -> list:
    return [int(p) & 0xFFFFFFFF for p in parts]


def _row_blocks(rows: int, cols: int):
    per = max(1, _BLOCK_VALUES // max(1, cols))
    return [(r, min(rows, r + per)) for r in range(0, rows, per)]


def _outlier_multiplier(cols: int, key: list, frac: float = 0.001,
                        factor: float = 20.0) -> np.ndarray:
    """Multiplier per input column: `factor` on round(frac*cols) (>= 1) seeded columns."""
    k = max(1, int(round(frac * cols)))
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(key + [0x0C07])))
    cols_sel = g.choice(cols, size=k, replace=False)
    m = np.ones(cols, dtype=np.float32)
    m[cols_sel] = factor
    return m


def normal_weight(rows: int, cols: int, sigma: float, key: list,
                  outliers: bool = False, mean: float = 0.0) -> np.ndarray:
    """float32 [rows, cols] of Normal(mean, sigma), optional outlier columns."""
    out = np.empty((rows, cols), dtype=np.float32)
    mult = _outlier_multiplier(cols, key) if outliers else None

    def fill(ib):
        i, (r0, r1) = ib
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(key + [i])))
        blk = out[r0:r1]
        g.standard_normal(out=blk.reshape(-1), dtype=np.float32)
        blk *= np.float32(sigma)
        if mean:
            blk += np.float32(mean)
        if mult is not None:
            blk *= mult

    _pool_map(fill, enumerate(_row_blocks(rows, cols)))
    return out


def student_t_weight(rows: int, cols: int, nu: float, scale: float,
                     key: list) -> np.ndarray:
    out = np.empty((rows, cols), dtype=np.float32)

    def fill(ib):
        i, (r0, r1) = ib
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(key + [i])))
        out[r0:r1] = (g.standard_t(nu, size=(r1 - r0, cols)) * scale).astype(np.float32)

    _pool_map(fill, enumerate(_row_blocks(rows, cols)))
    return out


def to_bf16(w: np.ndarray) -> np.ndarray:
    flat = w.reshape(-1)
    out = np.empty(flat.size, dtype=np.uint16)
    step = 1 << 22

    def conv(lo):
        out[lo:lo + step] = f32_to_bf16_bits(flat[lo:lo + step])

    _pool_map(conv, range(0, flat.size, step))
    return out.reshape(w.shape)


def quant_int4(w: np.ndarray, group: int = 128):
    """Symmetric per-group int4 codes (packed nibbles) and fp16 scales."""
    rows, cols = w.shape
    assert cols % group == 0 and cols % 2 == 0
    packed = np.empty((rows, cols // 2), dtype=np.uint8)
    scales = np.empty((rows, cols // group), dtype=np.float16)

    def q(rr):
        r0, r1 = rr
        g = w[r0:r1].reshape(r1 - r0, cols // group, group)
        amax = np.abs(g).max(axis=2)
        s16 = (amax / np.float32(7.0)).astype(np.float16)
        s16[s16 == 0] = np.float16(1.0)
        scales[r0:r1] = s16
        qq = np.rint(g / s16.astype(np.float32)[..., None])
        qq = np.clip(qq, -8, 7).astype(np.int8).reshape(r1 - r0, cols)
        nib = (qq.view(np.uint8) & 0x0F)
        packed[r0:r1] = nib[:, 0::2] | (nib[:, 1::2] << 4)

    _pool_map(q, _row_blocks(rows, cols))
    return packed, scales.view(np.uint16)


def quant_int8_rows(w: np.ndarray):
    """Per-output-row symmetric int8 codes and fp16 scales."""
    rows, cols = w.shape
    codes = np.empty((rows, cols), dtype=np.int8)
    scales = np.empty(rows, dtype=np.float16)

    def q(rr):
        r0, r1 = rr
        blk = w[r0:r1]
        amax = np.abs(blk).max(axis=1)
        s16 = (amax / np.float32(127.0)).astype(np.float16)
        s16[s16 == 0] = np.float16(1.0)
        scales[r0:r1] = s16
        qq = np.rint(blk / s16.astype(np.float32)[:, None])
        codes[r0:r1] = np.clip(qq, -127, 127).astype(np.int8)

    _pool_map(q, _row_blocks(rows, cols))
    return codes.view(np.uint8), scales.view(np.uint16)


def quant_fp8_rows(w: np.ndarray, fmt: str = "e4m3"):
    """Per-output-row scaled fp8 codes (OCP e4m3 'fn' or e5m2) and bf16 scales.

    scale = absmax_row / max_finite (448 for e4m3, 57344 for e5m2); the codes
    are torch's round-to-nearest-even conversion of w / scale.
    """
    import torch
    dt, fmax = {"e4m3": (torch.float8_e4m3fn, 448.0), "e5m2": (torch.float8_e5m2, 57344.0)}[fmt]
    rows, cols = w.shape
    codes = np.empty((rows, cols), dtype=np.uint8)
    scales = np.empty(rows, dtype=np.float32)

    def q(rr):
        r0, r1 = rr
        blk = torch.from_numpy(np.ascontiguousarray(w[r0:r1]))
        amax = blk.abs().amax(dim=1)
        sc = torch.where(amax > 0, amax / fmax, torch.ones_like(amax))
        scales[r0:r1] = sc.numpy()
        codes[r0:r1] = (blk / sc[:, None]).to(dt).view(torch.uint8).numpy()

    _pool_map(q, _row_blocks(rows, cols))
    return codes, to_bf16(scales)


_E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float32)


_E2M1_MID = (_E2M1[1:] + _E2M1[:-1]) / 2


def fp4_e2m1_codes(x: np.ndarray) -> np.ndarray:
    """4-bit e2m1 codes (sign << 3 | magnitude index) of x, round to nearest,
    ties to the even code, saturating at 6."""
    a = np.minimum(np.abs(x), np.float32(6.0))
    lo = np.searchsorted(_E2M1_MID, a, side="left")    # midpoints strictly below a
    hi = np.searchsorted(_E2M1_MID, a, side="right")   # midpoints at or below a
    idx = np.where(lo == hi, lo, np.where(lo % 2 == 0, lo, hi)).astype(np.uint8)
    sign = (np.signbit(x) & (idx > 0)).astype(np.uint8)
    return (sign << 3) | idx


def quant_mxfp4(w: np.ndarray, block: int = 32):
    """MXFP4 (OCP microscaling): e2m1 codes, packed two per byte (low nibble =
    even element), and one e8m0 scale byte per `block` inputs:
    scale = 2^(floor(log2(amax)) - 2), stored as its biased exponent."""
    rows, cols = w.shape
    assert cols % block == 0
    packed = np.empty((rows, cols // 2), dtype=np.uint8)
    scales = np.empty((rows, cols // block), dtype=np.uint8)

    def q(rr):
        r0, r1 = rr
        g = w[r0:r1].reshape(r1 - r0, cols // block, block)
        amax = np.abs(g).max(axis=2)
        e = np.where(amax > 0, np.floor(np.log2(np.maximum(amax, 1e-30))) - 2, -127)
        e = np.clip(e, -127, 127).astype(np.int32)
        scales[r0:r1] = (e + 127).astype(np.uint8)
        x = g / np.exp2(e.astype(np.float32))[..., None]
        c = fp4_e2m1_codes(x).reshape(r1 - r0, cols)
        packed[r0:r1] = c[:, 0::2] | (c[:, 1::2] << 4)

    _pool_map(q, _row_blocks(rows, cols))
    return packed, scales


def quant_awq4(w: np.ndarray, group: int = 128):
    """Asymmetric per-group 4-bit codes with zero points (AWQ-style storage):
    scale = (max - min) / 15 (fp16), zero = clamp(rint(-min / scale), 0, 15),
    q = clamp(rint(w / scale) + zero, 0, 15).  Codes and zeros are packed
    nibbles (low nibble = even element)."""
    rows, cols = w.shape
    assert cols % group == 0 and (cols // group) % 2 == 0
    packed = np.empty((rows, cols // 2), dtype=np.uint8)
    zeros = np.empty((rows, cols // group // 2), dtype=np.uint8)
    scales = np.empty((rows, cols // group), dtype=np.float16)

    def q(rr):
        r0, r1 = rr
        g = w[r0:r1].reshape(r1 - r0, cols // group, group)
        lo, hi = g.min(axis=2), g.max(axis=2)
        s16 = ((hi - lo) / np.float32(15.0)).astype(np.float16)
        s16[s16 == 0] = np.float16(1.0)
        s32 = s16.astype(np.float32)
        z = np.clip(np.rint(-lo / s32), 0, 15).astype(np.uint8)
        qq = np.clip(np.rint(g / s32[..., None]) + z[..., None], 0, 15).astype(np.uint8)
        qq = qq.reshape(r1 - r0, cols)
        packed[r0:r1] = qq[:, 0::2] | (qq[:, 1::2] << 4)
        zeros[r0:r1] = z[:, 0::2] | (z[:, 1::2] << 4)
        scales[r0:r1] = s16

    _pool_map(q, _row_blocks(rows, cols))
    return packed, zeros, scales.view(np.uint16)


# --------------------------------------------------------------------------
# Layer shapes ([out, in], PyTorch Linear layout).

LLAMA3_8B = [("q_proj", 4096, 4096), ("k_proj", 1024, 4096),
             ("v_proj", 1024, 4096), ("o_proj", 4096, 4096),
             ("gate_proj", 14336, 4096), ("up_proj", 14336, 4096),
             ("down_proj", 4096, 14336)]
LLAMA3_8B_NORMS = [("input_layernorm", 4096), ("post_attention_layernorm", 4096)]

LLAMA3_70B = [("q_proj", 8192, 8192), ("k_proj", 1024, 8192),
              ("v_proj", 1024, 8192), ("o_proj", 8192, 8192),
              ("gate_proj", 28672, 8192), ("up_proj", 28672, 8192),
              ("down_proj", 8192, 28672)]


def _scaled(shapes, div):
    if div == 1:
        return list(shapes)
    out = []
    for name, o, i in shapes:
        o2 = max(8, o // div)
        i2 = max(256, (i // div) // 256 * 256)
        out.append((name, o2, i2))
    return out


def _norms(seed: int, div: int):
    ts = []
    for j, (name, n) in enumerate(LLAMA3_8B_NORMS):
        n2 = max(64, n // div)
        w = normal_weight(1, n2, 0.02, _key(seed, 100 + j), mean=1.0)
        ts.append(Tensor(name, "bf16", to_bf16(w).reshape(n2), (n2,)))
    return ts


def config(cfg: int, layer: int = 0, div: int = 1) -> list:
    """Tensors of workload `cfg` (1..9).

    `div` > 1 shrinks every matrix dimension by that factor (same recipe,
    same distribution) so CPU-only tests stay fast; `layer` selects the
    layer seed of the 70B workload.
    """
    if cfg == 1:
        rows, cols = (4096 // div, 4096 // div) if div > 1 else (4096, 4096)
        w = normal_weight(rows, cols, 0.02, _key(0, 0))
        return [Tensor("weight", "bf16", to_bf16(w), (rows, cols))]
    if cfg == 2:
        ts = []
        for j, (name, o, i) in enumerate(_scaled(LLAMA3_8B, div)):
            w = normal_weight(o, i, 0.02, _key(1, j), outliers=True)
            ts.append(Tensor(name, "bf16", to_bf16(w), (o, i)))
        return ts + _norms(1, div)
    if cfg == 3:
        ts = []
        for j, (name, o, i) in enumerate(_scaled(LLAMA3_8B, div)):
            w = normal_weight(o, i, 0.02, _key(2, j))
            codes, scales = quant_int4(w)
            ts.append(Tensor(name + ".qweight", "u4", codes.reshape(-1), (o, i)))
            ts.append(Tensor(name + ".scales", "fp16", scales.reshape(-1), (o, i // 128)))
        return ts + _norms(2, div)
    if cfg == 4:
        ts = []
        for j, (name, o, i) in enumerate(_scaled(LLAMA3_8B, div)):
            w = student_t_weight(o, i, 5.0, 0.02, _key(3, j))
            codes, scales = quant_int8_rows(w)
            ts.append(Tensor(name + ".qweight", "u8", codes.reshape(-1), (o, i)))
            ts.append(Tensor(name + ".scales", "fp16", scales.reshape(-1), (o,)))
        return ts + _norms(3, div)
    if cfg == 5:
        ts = []
        for j, (name, o, i) in enumerate(_scaled(LLAMA3_70B, div)):
            w = normal_weight(o, i, 0.015, _key(4, layer, j), outliers=True)
            ts.append(Tensor(name, "bf16", to_bf16(w), (o, i)))
        return ts
    if cfg == 6:
        ts = []
        for j, (name, o, i) in enumerate(_scaled(LLAMA3_8B, div)):
            w = normal_weight(o, i, 0.02, _key(6, j), outliers=True)
            codes, scales = quant_fp8_rows(w, "e4m3")
            ts.append(Tensor(name + ".weight", "fp8_e4m3", codes.reshape(-1), (o, i)))
            ts.append(Tensor(name + ".scale", "bf16", scales.reshape(-1), (o,)))
        return ts + _norms(6, div)
    if cfg == 9:
        ts = []
        for j, (name, o, i) in enumerate(_scaled(LLAMA3_8B, div)):
            w = normal_weight(o, i, 0.02, _key(9, j), outliers=True)
            codes, scales = quant_fp8_rows(w, "e5m2")
            ts.append(Tensor(name + ".weight", "fp8_e5m2", codes.reshape(-1), (o, i)))
            ts.append(Tensor(name + ".scale", "bf16", scales.reshape(-1), (o,)))
        return ts + _norms(9, div)
    if cfg == 7:
        ts = []
        for j, (name, o, i) in enumerate(_scaled(LLAMA3_8B, div)):
            w = normal_weight(o, i, 0.02, _key(7, j), outliers=True)
            codes, scales = quant_mxfp4(w)
            ts.append(Tensor(name + ".blocks", "fp4_e2m1", codes.reshape(-1), (o, i)))
            ts.append(Tensor(name + ".scales", "u8", scales.reshape(-1), (o, i // 32)))
        return ts + _norms(7, div)
    if cfg == 8:
        ts = []
        for j, (name, o, i) in enumerate(_scaled(LLAMA3_8B, div)):
            w = normal_weight(o, i, 0.02, _key(8, j))
            codes, zeros, scales = quant_awq4(w)
            ts.append(Tensor(name + ".qweight", "u4", codes.reshape(-1), (o, i)))
            ts.append(Tensor(name + ".qzeros", "u4", zeros.reshape(-1), (o, i // 128)))
            ts.append(Tensor(name + ".scales", "fp16", scales.reshape(-1), (o, i // 128)))
        return ts + _norms(8, div)
    raise ValueError(f"unknown workload {cfg}")


CONFIG_NAMES = {
    1: "bf16 4096x4096 N(0,0.02)",
    2: "Llama-3-8B layer bf16 (outlier channels)",
    3: "Llama-3-8B layer int4 g128 + fp16 scales",
    4: "Llama-3-8B layer int8 per-row (Student-t nu=5) + fp16 scales",
    5: "Llama-3-70B layer bf16 (outlier channels)",
    6: "Llama-3-8B layer fp8 e4m3, per-row bf16 scales (outlier channels)",
    7: "Llama-3-8B layer MXFP4: e2m1 codes + e8m0 scales per 32 inputs",
    8: "Llama-3-8B layer AWQ-style int4 g128: codes + 4-bit zero points + fp16 scales",
    9: "Llama-3-8B layer fp8 e5m2, per-row bf16 scales (outlier channels)",
}


def _decoder_layer(d: int, f: int, kv: int, experts: int = 1, head: int = 128):
    """Linear shapes of one decoder layer: hidden size d, intermediate size f,
    kv key/value heads of `head` dims (grouped-query attention), `experts`
    MLP experts."""
    shapes = [("q_proj", d, d), ("k_proj", kv * head, d), ("v_proj", kv * head, d),
              ("o_proj", d, d)]
    for e in range(experts):
        p = f"experts.{e}." if experts > 1 else ""
        shapes += [(p + "gate_proj", f, d), (p + "up_proj", f, d), (p + "down_proj", d, f)]
    return shapes


# One bf16 decoder layer of each model family the paper evaluates (Sec. VI-A,
# 1.5B to 405B parameters), with the sizes of the public model configurations,
# and the sigma of the Normal draw (0.1 % outlier input columns x20 as above).
MODEL_LAYERS = {
    "qwen2-1.5b": (_decoder_layer(1536, 8960, 2), 0.02),
    "mistral-7b": (_decoder_layer(4096, 14336, 8), 0.02),
    "qwen2.5-14b": (_decoder_layer(5120, 13824, 8), 0.02),
    "deepseek-67b": (_decoder_layer(8192, 22016, 8), 0.015),
    "mixtral-8x22b": (_decoder_layer(6144, 16384, 8, experts=8), 0.015),
    "llama3-405b": (_decoder_layer(16384, 53248, 8), 0.01),
}


def layer_torch_device(shapes, sigma: float, seed: int, layer: int = 0, device: str = "cuda"):
    """bf16 Normal(0, sigma) tensors with 0.1 % outlier input columns x20, drawn
    on the GPU with torch's Philox generator seeded (seed, layer, tensor).
    Returns a list of (name, uint8 device tensor holding the bf16 storage,
    shape)."""
    import torch
    out = []
    for j, (name, o, i) in enumerate(shapes):
        g = torch.Generator(device=device)
        g.manual_seed((seed << 40) | (layer << 20) | j)
        w = torch.randn((o, i), generator=g, device=device, dtype=torch.float32)
        w.mul_(sigma)
        mult = torch.from_numpy(_outlier_multiplier(i, _key(seed, layer, j))).to(device)
        w.mul_(mult)
        b = w.to(torch.bfloat16)
        del w
        out.append((name, b.view(torch.uint8).reshape(-1), (o, i)))
    return out


def int8_rows_torch_device(rows: int, cols: int, seed: int, device: str = "cuda",
                           block_rows: int = 4096):
    """Per-row symmetric int8 codes of Normal(0, 1) draws on the GPU: scale =
    absmax(row) / 127, q = round(w / scale), stored as uint8 (two's complement).
    Row block b is drawn with torch's Philox generator seeded (seed, b).
    Returns a uint8 device tensor of rows * cols bytes."""
    import torch
    out = torch.empty(rows * cols, dtype=torch.uint8, device=device)
    for b, r0 in enumerate(range(0, rows, block_rows)):
        r1 = min(rows, r0 + block_rows)
        g = torch.Generator(device=device)
        g.manual_seed((seed << 40) | b)
        w = torch.randn((r1 - r0, cols), generator=g, device=device, dtype=torch.float32)
        scale = w.abs().amax(dim=1, keepdim=True).clamp_min(1e-30) / 127.0
        q = torch.round(w / scale).clamp_(-127, 127).to(torch.int8)
        out[r0 * cols:r1 * cols] = q.view(torch.uint8).reshape(-1)
        del w, q
    return out


def config_torch_device(cfg: int, layer: int, device: str = "cuda"):
    """70B-layer bf16 tensors drawn on the GPU with torch's device generator.

    Same shapes and statistics as ``config(5, layer)``; the draw itself comes
    from torch's Philox stream seeded with (4, layer, tensor), so values
    differ from the numpy recipe.  Returns a list of (name, uint8 device
    tensor holding the bf16 storage, shape).
    """
    if cfg != 5:
        raise ValueError("device-side drawing is provided for the 70B layer only")
    return layer_torch_device(LLAMA3_70B, 0.015, 4, layer, device)
