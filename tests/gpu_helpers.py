"""Shared pieces of the GPU tests: layers on the device, conversions between
bf16 bit patterns and values, the oracle side of each comparison, and the
parity bar (max-abs 2e-2 and relative Frobenius 1e-2 against the oracle)."""
import functools
import sys

import numpy as np
import torch

from oracle import layer as O
from paper_2607_15865_amd import synth

MAX_ABS = 2e-2
REL_FRO = 1e-2


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=4)
def host_layer(name: str, layer: int = 0, with_zeros: bool = False):
    cfg = synth.CONFIGS[name]
    w = synth.make_layer(cfg, layer, with_zeros)
    return cfg, w


@functools.lru_cache(maxsize=2)
def oracle_weights(name: str, layer: int = 0, with_zeros: bool = False):
    cfg, w = host_layer(name, layer, with_zeros)
    return O.dequant_layer(w, cfg)


_dev_layers = {}


def device_layer(name: str, layer: int = 0, with_zeros: bool = False):
    from paper_2607_15865_amd import binding
    key = (name, layer, with_zeros)
    if key not in _dev_layers:
        if len(_dev_layers) >= 3:
            _dev_layers.pop(next(iter(_dev_layers))).close()
        cfg, w = host_layer(name, layer, with_zeros)
        _dev_layers[key] = binding.Layer(cfg, w)
    return _dev_layers[key]


def bits_to_torch_f32(bits: np.ndarray) -> torch.Tensor:
    """bf16 bit patterns -> float32 tensor on the GPU (exact)."""
    u = bits.astype(np.uint32) << 16
    return torch.from_numpy(u.view(np.float32).copy()).cuda()


def cache_values(t: torch.Tensor) -> np.ndarray:
    """bf16 cache (int16 bit patterns) -> fp64 values on the host."""
    return O.bf16_to_f64(t.cpu().numpy().view(np.uint16))


def to_cache_bits(vals: np.ndarray) -> np.ndarray:
    """fp64 values that are bf16 numbers -> their bit patterns (int16)."""
    f = np.ascontiguousarray(vals.astype(np.float32))
    return (f.view(np.uint32) >> 16).astype(np.uint16).view(np.int16)


def assert_parity(got, ref, what: str):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - ref)
    mx = float(err.max()) if err.size else 0.0
    rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))
    log(f"  {what}: max-abs {mx:.3e}  rel-fro {rel:.3e}  (n={err.size})")
    assert mx <= MAX_ABS, f"{what}: max-abs {mx} > {MAX_ABS}"
    assert rel <= REL_FRO, f"{what}: rel-fro {rel} > {REL_FRO}"
    return mx, rel
