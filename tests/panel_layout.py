"""The library's panel-major buffer layout, as pure data movement (NumPy).

The oracle produces row-major packed buffers (codes, metadata and scales per
row, in the byte order of the method's compressed representation).  The HIP
library stores the same bytes panel-major: K is cut into panels of 128
positions (the last one may be narrower), panel p holds the bytes of all rows
for its K range, row after row, and panels follow each other.  These helpers
convert between the two; they hold none of the method's arithmetic, and the
oracle does not import them.
"""

from __future__ import annotations

import numpy as np

from oracle import sharq_oracle as O

PANEL_K = 128


def to_panels(rowmajor: np.ndarray, K: int) -> np.ndarray:
    """Row-major [R, bytes(K)] -> flat panel-major bytes (every buffer holds a
    fixed number of bytes per 32 K positions)."""
    a = np.asarray(rowmajor, dtype=np.uint8)
    R, B = a.shape
    per32 = B // (K // 32)
    parts = []
    for lo in range(0, K, PANEL_K):
        hi = min(lo + PANEL_K, K)
        parts.append(a[:, lo // 32 * per32: hi // 32 * per32].reshape(-1))
    return np.concatenate(parts) if parts else np.zeros(0, np.uint8)


def from_panels(flat: np.ndarray, R: int, K: int, bytes_per_row: int) -> np.ndarray:
    """Inverse of to_panels: flat panel-major bytes -> row-major [R, bytes_per_row]."""
    flat = np.asarray(flat, dtype=np.uint8).reshape(-1)
    per32 = bytes_per_row // (K // 32)
    out = np.zeros((R, bytes_per_row), dtype=np.uint8)
    off = 0
    for lo in range(0, K, PANEL_K):
        hi = min(lo + PANEL_K, K)
        w = (hi - lo) // 32 * per32
        out[:, lo // 32 * per32: hi // 32 * per32] = flat[off: off + R * w].reshape(R, w)
        off += R * w
    return out


def act_to_device_layout(act: dict) -> dict:
    """An oracle-prepared activation's buffers in the library's panel-major layout."""
    return {k: to_panels(act[k], act["K"]) for k in O.ACT_BUFFERS_ALL if k in act}


def act_from_device_layout(bufs: dict, rows: int, K: int, n: int, m: int, fmt: str, tensor_scale=None,
                           mode: str = "sharq", pairs: bool = False) -> dict:
    """Panel-major device buffers -> the row-major dict the oracle's GEMM reads."""
    widths = O.act_widths(K, n, m, fmt, mode)
    d = {"rows": rows, "K": K, "n": n, "m": m, "fmt": fmt, "tensor_scale": tensor_scale, "mode": mode,
         "pairs": pairs}
    for k in O.ACT_BUFFERS_ALL:
        if widths[k] == 0:
            d[k] = np.zeros((rows, 0), np.uint8)
        else:
            d[k] = from_panels(bufs[k], rows, K, widths[k])
    return d


def weight_to_device_layout(wq: dict) -> dict:
    return {k: to_panels(wq[k], wq["K"]) for k in O.WEIGHT_BUFFERS}


def weight_from_device_layout(bufs: dict, N: int, K: int, fmt: str, tensor_scale=None) -> dict:
    widths = {"codes": K // 2, "scale": K // 16 if fmt == "hif4" else K // 32,
              "scale_dn": K // 32 if fmt == "mx" else K // 16}
    d = {"N": N, "K": K, "fmt": fmt, "tensor_scale": tensor_scale}
    for k in O.WEIGHT_BUFFERS:
        d[k] = from_panels(bufs[k], N, K, widths[k])
    return d


def dense_backbone_rowmajor(act: dict) -> np.ndarray:
    """The library's optional dense backbone copy of an oracle-prepared
    activation: the backbone's E2M1 codes at every K position (dropped
    positions code 0), two per byte, row-major [rows, K/2].  It is the oracle's
    compressed backbone expanded back to K positions."""
    dense, _ = O.unpack_backbone(act["sp_codes"], act["sp_meta"], act["K"], act["n"], act["m"])
    return O.pack_nibbles(dense)


def dense_backbone_to_device_layout(act: dict) -> np.ndarray:
    return to_panels(dense_backbone_rowmajor(act), act["K"])
