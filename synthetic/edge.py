"""Edge-case input recipes: the regular seeded inputs of a workload with some
tensors re-drawn or overwritten so that the degenerate cases of the method
occur.  Like the rest of this package it only builds input values (random
draws, constants, sign flips, scaling by a power of two) and rounds them to
the storage dtype; it computes nothing of the primitive graphs.

Cases (each at the workload's full size unless sizes are given):
  * conv / "wide_shift": the BatchNorm shift of channel j is -120 + 240 j /
    (Cout - 1), so the Mish argument sweeps [-121, 121]: arguments above 20
    (where tanh(softplus(x)) is 1 in fp32) and below -88 (where exp(x)
    underflows in fp32) both occur;
  * mlp / "flat_rows": rows 0-15 of X are constants (-3.0 ... +2.625 in steps
    of 0.375), row 16 is all zeros and row 17 alternates +1 / -1, so the
    LayerNorm variance of rows 0-16 is exactly zero (the row scale is
    1/sqrt(eps));
  * instnorm / "flat_channels": channels 0-3 of X are the constants 0.3, -1.5,
    0 and 2.25 over every pixel (zero InstanceNorm variance);
  * attention / "wide_scores" and sra / "wide_scores": Q (attention) or X
    (spatial-reduction attention, whose queries are the pixels) times 8, so
    the scores spread over several tens and most exponentials underflow;
  * linattn / "zero_rows": in every head the query rows t = 0, 7, 14, ... are
    made all-negative (their ReLU is zero, so their output is exactly 0), and
    every key of head 2 is negative (its key sums and K^T V are zero, so the
    whole head's output is exactly 0).
"""

from __future__ import annotations

import numpy as np

from . import bf16_bits_to_f32, round_to_storage
from . import workloads as W

CASES = {
    "conv": "wide_shift",
    "mlp": "flat_rows",
    "instnorm": "flat_channels",
    "attention": "wide_scores",
    "sra": "wide_scores",
    "linattn": "zero_rows",
}


def _f32(a, dtype):
    """Storage array -> float32 values (exact)."""
    return bf16_bits_to_f32(a) if dtype == "bf16" else np.asarray(a, dtype=np.float32)


def edge_inputs(workload: str, **sizes):
    """``{name: storage_array}`` of the workload's edge case (see the module
    docstring), built from the regular seeded inputs."""
    specs = W.specs(workload, **sizes)
    dtype = specs[0][3]
    raw = W.make_inputs(specs)
    x = {k: _f32(v, dtype).copy() for k, v in raw.items()}
    if workload == "conv":
        cout = x["shift"].shape[0]
        x["shift"] = (-120.0 + 240.0 * np.arange(cout) / max(cout - 1, 1)).astype(np.float32)
    elif workload == "mlp":
        m = x["X"].shape[0]
        for i in range(min(16, m)):
            x["X"][i, :] = -3.0 + 0.375 * i
        if m > 16:
            x["X"][16, :] = 0.0
        if m > 17:
            x["X"][17, :] = np.where(np.arange(x["X"].shape[1]) % 2 == 0, 1.0, -1.0)
    elif workload == "instnorm":
        for ch, v in enumerate((0.3, -1.5, 0.0, 2.25)):
            if ch < x["X"].shape[-1]:
                x["X"][..., ch] = v
    elif workload == "attention":
        x["Q"] *= 8.0
    elif workload == "sra":
        x["X"] *= 8.0
    elif workload == "linattn":
        x["Q"][:, ::7, :] = -np.abs(x["Q"][:, ::7, :])
        if x["K"].shape[0] > 2:
            x["K"][2] = -np.abs(x["K"][2])
    else:
        raise ValueError(workload)
    # every change above keeps values representable in the storage dtype
    # (constants with few significant bits, sign flips, power-of-two scaling),
    # except the conv shift, which is rounded here like any drawn value
    return {k: round_to_storage(v, dtype) for k, v in x.items()}
