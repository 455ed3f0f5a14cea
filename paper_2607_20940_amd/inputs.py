"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke
check.

This module holds no MSSA arithmetic: it turns (shapes, seed, amplitude,
dtype) into input bytes and converts storage formats.  Token counts are
passed in by the caller.

Recipe: ``numpy.random.default_rng(seed).standard_normal(shape)`` in float64,
drawn tensor by tensor in the order of ``DRAW_ORDER`` (empty tensors are
skipped and draw nothing), multiplied by the amplitude, rounded to float32
(round-to-nearest-even) and, for bf16, from float32 to bf16
(round-to-nearest-even).  Those stored values are the inputs: the GPU gets
the bytes, the oracle gets the same values widened exactly to float64.
"""

import numpy as np

DRAW_ORDER = ("q_win", "k_win", "v_win", "k_sink", "v_sink", "k_hist", "v_hist")


def f32_to_bf16_bits(x32):
    """float32 array -> uint16 bf16 bit patterns, round-to-nearest-even
    (inputs are finite)."""
    b = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    rounded = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(u16):
    u = np.ascontiguousarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32)


def to_f64(x, dtype):
    """Stored input (uint16 bf16 bits or float32) -> float64, exactly."""
    if x is None:
        return None
    if dtype == "bf16":
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def make_inputs(shapes, seed, amplitude=1.0, dtype="bf16", q_amplitude=None):
    """shapes: mapping name -> shape tuple for the names in DRAW_ORDER (a
    missing or zero-sized entry is empty).  Returns name -> stored array
    (uint16 bf16 bits, or float32), None for empty tensors.  q_amplitude, if
    given, replaces the amplitude of q_win (the draws are the same)."""
    rng = np.random.default_rng(seed)
    out = {}
    for name in DRAW_ORDER:
        shape = tuple(shapes.get(name, (0,)))
        if int(np.prod(shape)) == 0:
            out[name] = None
            continue
        amp = q_amplitude if (name == "q_win" and q_amplitude is not None) else amplitude
        x = (rng.standard_normal(shape) * amp).astype(np.float32)
        out[name] = f32_to_bf16_bits(x) if dtype == "bf16" else x
    return out


def make_grad_output(shape, seed, amplitude=1.0, dtype="bf16"):
    """Seeded gradient of the attention output (same recipe as the inputs:
    N(0, 1) draws times the amplitude, rounded once to the dtype)."""
    x = (np.random.default_rng(seed).standard_normal(tuple(shape)) * amplitude).astype(np.float32)
    return f32_to_bf16_bits(x) if dtype == "bf16" else x


def make_inputs_device(shapes, seed, amplitude=1.0, dtype="bf16", names=DRAW_ORDER, device="cuda",
                       q_amplitude=None):
    """Device-side variant for workloads too large to draw on the host:
    torch's generator on `device` seeded with `seed` draws N(0,1) float32
    tensors in the order of `names`, scaled by the amplitude (q_amplitude
    for q_win if given) and rounded to bf16 (round-to-nearest-even) or kept
    float32.  The values are defined by this function (the oracle reads them
    back from the device)."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    out = {}
    for name in names:
        shape = tuple(shapes.get(name, (0,)))
        if int(np.prod(shape)) == 0:
            out[name] = None
            continue
        amp = q_amplitude if (name == "q_win" and q_amplitude is not None) else amplitude
        x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32) * amp
        out[name] = x.to(torch.bfloat16) if dtype == "bf16" else x
    return out
