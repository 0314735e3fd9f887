"""Seeded synthetic activations shaped like the paper's workloads.

This module holds no arithmetic of the method: it only draws random numbers,
rounds them to bf16 and returns bit patterns.  Both the HIP path (tests,
benchmark) and the CPU oracle (tests) take their inputs from here.

The paper benchmarks its kernels on random Gaussian inputs over Llama-3 hidden
sizes (appendix "Performance Benchmark Details"); its training activations
came from a text corpus that is not used here.  The presets below stand in for
those activations: Gaussian rows, rows with a per-token scale, rows with
outlier feature channels (the outlier features of Sec. 4.3), and a heavy-tailed
stress case with saturating elements, all-zero rows and constant rows.

Recipe (every preset):
  * rows are drawn in chunks of ``CHUNK`` rows; chunk c uses
    ``numpy.random.default_rng([seed, c])`` so any row range can be rebuilt
    without drawing the whole tensor;
  * per-tensor choices (outlier channels, gain, special rows) come from
    ``default_rng([seed, AUX])``, drawn in the order: channel/row modifiers,
    then the gain;
  * float32 values are rounded to bf16 with round-to-nearest-even.
"""
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

CHUNK = 4096
AUX = 1 << 30


def f32_to_bf16_bits(x):
    """Round float32 values to bf16 (nearest, ties to even); NaN stays NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    nan = np.isnan(x)
    # no uint32 overflow: finite and infinite patterns are <= 0xFF800000
    r = np.where(nan, np.uint32(0), u)
    r = (r + ((r >> 16) & 1) + np.uint32(0x7FFF)) >> 16
    out = r.astype(np.uint16)
    if nan.any():
        out[nan] = ((u[nan] >> 16) | 0x40).astype(np.uint16)
    return out


def bf16_bits_to_f32(b):
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class Preset:
    name: str
    T: int
    d: int
    fmt: str           # "mxfp8" or "nvfp4"
    kind: str          # generator kind, see _draw_chunk
    gamma: str         # "normal" (1 + 0.1 N(0,1)) or "uniform" (U[0.5, 1.5])
    description: str = field(default="", compare=False)


PRESETS = {
    p.name: p
    for p in [
        Preset("llama3-125m-d768", 1024, 768, "mxfp8", "gauss", "normal",
               "x ~ N(0,1) [1024, 768]; gamma = 1 + 0.1 N(0,1)"),
        Preset("llama3-1b-d2048", 16384, 2048, "mxfp8", "gauss_rowscale", "normal",
               "x ~ N(0,1) * s_t, s_t log-uniform in [0.1, 10] per row [16384, 2048]"),
        Preset("llama3-8b-d4096", 32768, 4096, "mxfp8", "gauss_outlier", "normal",
               "x ~ N(0,1) [32768, 4096] with 41 (1%) channels x20 as outlier features"),
        Preset("llama3-8b-d4096-nvfp4", 32768, 4096, "nvfp4", "gauss_outlier", "normal",
               "same x as llama3-8b-d4096; NVFP4 output"),
        Preset("llama3-8b-longctx-stress", 131072, 4096, "mxfp8", "t3_stress", "uniform",
               "x ~ t(3)/sqrt(3) [131072, 4096]; 0.1% elements = +-448; 1% zero rows, "
               "1% constant rows; gamma ~ U[0.5, 1.5]"),
    ]
}


def _aux(preset, seed):
    """Per-tensor modifiers, drawn in a fixed order from one generator."""
    rng = np.random.default_rng([seed, AUX])
    aux = {}
    if preset.kind == "gauss_outlier":
        n = int(round(0.01 * preset.d))
        aux["outlier_channels"] = np.sort(rng.choice(preset.d, n, replace=False))
    if preset.kind == "t3_stress":
        perm = rng.permutation(preset.T)
        n = preset.T // 100
        aux["zero_rows"] = np.sort(perm[:n])
        const_rows = perm[n:2 * n]
        order = np.argsort(const_rows)
        aux["const_rows"] = const_rows[order]
        aux["const_values"] = rng.standard_normal(n).astype(np.float32)[order]
    if preset.gamma == "normal":
        aux["gamma"] = (1.0 + 0.1 * rng.standard_normal(preset.d)).astype(np.float32)
    else:
        aux["gamma"] = rng.uniform(0.5, 1.5, preset.d).astype(np.float32)
    return aux


def _draw_chunk(preset, seed, c, aux):
    r0 = c * CHUNK
    r1 = min(preset.T, r0 + CHUNK)
    n = r1 - r0
    rng = np.random.default_rng([seed, c])
    d = preset.d
    if preset.kind in ("gauss", "gauss_rowscale", "gauss_outlier"):
        x = rng.standard_normal((n, d), dtype=np.float32)
        if preset.kind == "gauss_rowscale":
            s = np.exp(rng.uniform(np.log(0.1), np.log(10.0), n)).astype(np.float32)
            x *= s[:, None]
        elif preset.kind == "gauss_outlier":
            x[:, aux["outlier_channels"]] *= np.float32(20.0)
    elif preset.kind == "t3_stress":
        # Student t with 3 degrees of freedom, Z / sqrt(V / 3) with V the sum
        # of three squared normals, scaled by 1/sqrt(3) to unit variance
        z = rng.standard_normal((n, d), dtype=np.float32)
        v = np.zeros((n, d), np.float32)
        for _ in range(3):
            w = rng.standard_normal((n, d), dtype=np.float32)
            v += w * w
        x = z / np.sqrt(v)
        hit = rng.random((n, d)) < 0.001
        sign = np.where(rng.random((n, d)) < 0.5, -1.0, 1.0).astype(np.float32)
        x[hit] = 448.0 * sign[hit]
        zr = aux["zero_rows"]
        zr = zr[(zr >= r0) & (zr < r1)] - r0
        x[zr] = 0.0
        cr = aux["const_rows"]
        sel = (cr >= r0) & (cr < r1)
        x[cr[sel] - r0] = aux["const_values"][sel][:, None]
    else:
        raise ValueError(preset.kind)
    return x


@dataclass
class Workload:
    preset: Preset
    x: np.ndarray          # uint16 bf16 bits [rows, d]
    gamma: np.ndarray      # uint16 bf16 bits [d]
    rows: np.ndarray       # the row indices of the full tensor that x holds


def generate(name, seed=0, rows=None):
    """Build preset ``name``.  ``rows`` (sorted indices) selects a subset of
    the full tensor's rows -- the same values the full tensor holds there."""
    preset = PRESETS[name]
    aux = _aux(preset, seed)
    if rows is None:
        rows = np.arange(preset.T)
    rows = np.asarray(rows, dtype=np.int64)
    if rows.size and (rows.min() < 0 or rows.max() >= preset.T):
        raise ValueError("row index out of range")
    out = np.empty((rows.size, preset.d), np.uint16)
    chunks = np.unique(rows // CHUNK)

    def fill(c):
        x = _draw_chunk(preset, seed, int(c), aux)
        sel = np.nonzero(rows // CHUNK == c)[0]
        out[sel] = f32_to_bf16_bits(x[rows[sel] - c * CHUNK])

    # chunks are independent streams; threads only change the wall time
    with ThreadPoolExecutor(max_workers=min(8, len(chunks)) or 1) as ex:
        list(ex.map(fill, chunks))
    return Workload(preset, out, f32_to_bf16_bits(aux["gamma"]), rows)


def gaussian(T, d, seed=0, scale=1.0):
    """Plain N(0, scale^2) bf16 rows for tests of arbitrary shape."""
    rng = np.random.default_rng([seed, 7])
    return f32_to_bf16_bits(scale * rng.standard_normal((T, d), dtype=np.float32))
