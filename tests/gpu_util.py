"""Helpers shared by the GPU tests: move seeded inputs and oracle buffers
between NumPy and the device, and rebuild oracle-shaped dicts from device
buffers.  No arithmetic of the method lives here."""

import numpy as np
import torch

from oracle import sharq_oracle as O
import panel_layout as L
from paper_2606_26587_amd import sharq as S


def dev_bf16(u16: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).cuda()


def dev_u8(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8)).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


FMT_NAME = {S.MXFP4: "mx", S.NVFP4: "nv", S.HIF4: "hif4"}
FMT_ID = {"mx": S.MXFP4, "nv": S.NVFP4, "hif4": S.HIF4}
MODE_NAME = {v: k for k, v in S.MODES.items()}


def act_to_oracle(a: S.PreparedAct) -> dict:
    """Device prepared activation -> the oracle's row-major dict."""
    bufs = {k: host(getattr(a, k)) for k in O.ACT_BUFFERS}
    if a.dn_meta is not None:
        bufs["dn_meta"] = host(a.dn_meta)
    ts = None if a.tensor_scale is None else np.float32(host(a.tensor_scale)[0])
    return L.act_from_device_layout(bufs, a.rows, a.K, a.n, a.m, FMT_NAME[a.fmt], ts, mode=MODE_NAME[a.mode],
                                    pairs=a.pairs)


def oracle_to_act(o: dict, dense_backbone: bool = False) -> S.PreparedAct:
    """Oracle prepared activation -> device buffers in the library's layout
    (dense_backbone: with the MXFP4 dense backbone copy as well)."""
    fmt = FMT_ID[o["fmt"]]
    dev = L.act_to_device_layout(o)
    spd = dev_u8(L.dense_backbone_to_device_layout(o)) if dense_backbone else None
    ts = None
    if fmt == S.NVFP4:
        ts = torch.tensor([float(o["tensor_scale"])], dtype=torch.float32, device="cuda")
    mode = S.MODES[o.get("mode", "sharq")]
    dn_meta = dev_u8(dev["dn_meta"]) if "dn_meta" in dev else None
    return S.PreparedAct(o["rows"], o["K"], fmt, o["n"], o["m"], dev_u8(dev["sp_codes"]),
                         dev_u8(dev["sp_meta"]), dev_u8(dev["sp_scale"]), dev_u8(dev["dn_codes"]),
                         dev_u8(dev["dn_scale"]), tensor_scale=ts, pairs=bool(o.get("pairs", False)), mode=mode,
                         dn_meta=dn_meta, sp_dense=spd)


def oracle_to_weight(o: dict) -> S.QuantWeight:
    fmt = FMT_ID[o["fmt"]]
    dev = L.weight_to_device_layout(o)
    codes = dev_u8(dev["codes"])[None]
    scale = dev_u8(dev["scale"])[None]
    scale_dn = scale if fmt != S.NVFP4 else dev_u8(dev["scale_dn"])[None]
    ts = None if fmt != S.NVFP4 else torch.tensor([float(o["tensor_scale"])], dtype=torch.float32, device="cuda")
    return S.QuantWeight(o["N"], o["K"], 1, fmt, codes, scale, scale_dn, ts)


def weight_to_oracle(w: S.QuantWeight, e: int = 0) -> dict:
    bufs = {"codes": host(w.codes[e]), "scale": host(w.scale[e]), "scale_dn": host(w.scale_dn[e])}
    ts = None if w.tensor_scale is None else np.float32(host(w.tensor_scale)[e])
    return L.weight_from_device_layout(bufs, w.N, w.K, FMT_NAME[w.fmt], ts)


def assert_bytes_equal(name, got: np.ndarray, want: np.ndarray):
    got = np.asarray(got)
    want = np.asarray(want)
    assert got.shape == want.shape, (name, got.shape, want.shape)
    bad = np.nonzero(got != want)
    if bad[0].size:
        idx = tuple(b[0] for b in bad)
        raise AssertionError(f"{name}: {bad[0].size} of {got.size} bytes differ; first at {idx}: "
                             f"got {got[idx]:#x} want {want[idx]:#x}")
