"""Comparators between the HIP path and the oracle (test helpers).

Tolerances (derived from the arithmetic; the same readings are listed with
the design notes):
  * ids: equal rank by rank, except where the two facts' exact scores differ
    by less than 1e-6 (a near tie the fp32 scan may order either way);
  * scores: |s_gpu - s*| <= 1e-5 |s*|, or <= 2^-20 * sum_t |q_t e_t|: 16 fp32
    units in the last place of the magnitude sum, the first-order error bound
    of an fp32 reduction 16 additions deep, which covers scores near zero
    where cancellation makes any relative bound unreachable (the exact
    scores come from the oracle, the magnitudes from the decoded inputs);
  * slots, positions, m, V pages: bit-exact;
  * rotated keys: at most 1 bf16 ulp apart, or within 2^-7 relative, or
    within 2^-20 of the rotation pair's norm (an output that nearly cancels
    inherits the fp32 rounding of the norm, not of itself); and at most 0.1%
    of them may differ at all (only values next to a rounding boundary can).
"""
from __future__ import annotations

import numpy as np

import oracle

SENTINEL = 0x7FA5


def ordered_bf16(bits: np.ndarray) -> np.ndarray:
    b = bits.astype(np.int64)
    mag = b & 0x7FFF
    return np.where(b & 0x8000, -mag, mag)


def check_ids(gpu_ids: np.ndarray, ora_ids: np.ndarray, s_star: np.ndarray, n: int):
    """gpu_ids/ora_ids [k]; s_star [n] exact scores of that query."""
    assert len(set(gpu_ids.tolist())) == gpu_ids.size, "duplicate ids"
    assert (gpu_ids >= 0).all() and (gpu_ids < n).all(), "id out of range"
    diff = gpu_ids != ora_ids
    if diff.any():
        gap = np.abs(s_star[gpu_ids[diff]] - s_star[ora_ids[diff]])
        assert (gap < 1e-6).all(), f"rank mismatch beyond near ties: max gap {gap.max()}"
    return int(diff.sum())


def check_scores(gpu_scores: np.ndarray, s_star: np.ndarray, mag: np.ndarray) -> int:
    """gpu_scores [k] against the exact scores s_star [k] of the same facts;
    mag [k] = sum_t |q_t e_t| of each fact from the decoded (float) values.
    Returns how many scores needed the absolute floor."""
    mag = np.asarray(mag)
    assert mag.dtype.kind == "f" and np.asarray(s_star).dtype.kind == "f", \
        "magnitudes and exact scores must be decoded values, not bit patterns"
    assert mag.shape == np.shape(gpu_scores) == np.shape(s_star)
    err = np.abs(gpu_scores.astype(np.float64) - s_star)
    rel_ok = err <= 1e-5 * np.abs(s_star)
    ok = rel_ok | (err <= 2.0 ** -20 * mag)
    assert ok.all(), f"score mismatch: worst {err[~ok].max()} at {np.nonzero(~ok)[0][:5]}"
    return int((~rel_ok).sum())


def check_k_rows(gpu_bits: np.ndarray, ora_bits: np.ndarray, pre_bits: np.ndarray, D: int,
                 interleaved: bool = False):
    """Rows [..., H*D] (or [..., H, D]) of rotated keys; pre_bits the
    unrotated input rows of the same shape; interleaved: pairs (2j, 2j+1)
    instead of (j, j + D/2). Returns the count of elements that needed the
    pair-norm floor."""
    g = gpu_bits.reshape(-1, D)
    o = ora_bits.reshape(-1, D)
    x = oracle.bf16_to_f64(pre_bits.reshape(-1, D))
    half = D // 2
    if interleaved:
        pn = np.hypot(x[:, 0::2], x[:, 1::2])
        pair = np.empty_like(x)
        pair[:, 0::2], pair[:, 1::2] = pn, pn
    else:
        pair = np.hypot(x[:, :half], x[:, half:])
        pair = np.concatenate([pair, pair], axis=1)
    if np.array_equal(g, o):
        return 0
    ulp = np.abs(ordered_bf16(g) - ordered_bf16(o))
    gv, ov = oracle.bf16_to_f64(g), oracle.bf16_to_f64(o)
    err = np.abs(gv - ov)
    rel_ok = err <= 2.0 ** -7 * np.abs(ov)
    floor_ok = err <= 2.0 ** -20 * pair
    ok = (ulp <= 1) | rel_ok | floor_ok
    bad = ~ok
    assert not bad.any(), (f"{int(bad.sum())} rotated-key elements out of tolerance; worst ulp "
                           f"{int(ulp[bad].max())}, e.g. gpu {gv[bad][:3]} vs oracle {ov[bad][:3]}")
    # fp32 rotation then round-to-nearest-even should differ from the exactly
    # rounded binary64 result only next to a rounding boundary: a truncating
    # or otherwise biased conversion would be off in a large fraction of
    # elements while staying within one ulp
    differ = float((g != o).mean())
    assert differ <= 1e-3, f"{differ:.2%} of rotated-key elements are not bit-exact"
    return int(((ulp > 1) & ~rel_ok & floor_ok).sum())
