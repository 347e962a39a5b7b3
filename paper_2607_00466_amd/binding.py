"""ctypes binding of libeldr_moe.so: argument marshalling only.

Each function has the name and argument order of the C entry point it wraps
(see include/eldr_moe.h); torch tensors stand in for device pointers and the
stream defaults to torch's current stream.  Every step of the layer runs in
the library's HIP kernels; there is no fallback, and a missing library or a
non-zero status raises.
"""
from __future__ import annotations

import ctypes
import os
import re
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libeldr_moe.so")
INCLUDE_DIR = os.path.join(os.path.dirname(_PKG), "include")
HEADER_PATH = os.path.join(INCLUDE_DIR, "eldr_moe.h")
HEADER_PATHS = (HEADER_PATH, os.path.join(INCLUDE_DIR, "eldr_signature.h"),
                os.path.join(INCLUDE_DIR, "eldr_calibration.h"),
                os.path.join(INCLUDE_DIR, "eldr_route.h"))

MOE_OK = 0
MOE_ERR_INVALID = -1
MOE_ERR_UNSUPPORTED = -2
MOE_ERR_WORKSPACE = -3
MOE_ERR_HIP = -4

# Shape limits of the layer calls (include/eldr_moe.h).
MOE_MAX_E = 256
MOE_MAX_K = 16
MOE_MAX_T = 4096
MOE_MAX_H = 16384
MOE_MAX_I = 16384


class MoeDims(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("H", ctypes.c_int32), ("E", ctypes.c_int32),
                ("K", ctypes.c_int32), ("I", ctypes.c_int32)]

    def __repr__(self) -> str:
        return f"MoeDims(T={self.T}, H={self.H}, E={self.E}, K={self.K}, I={self.I})"


class MoeError(RuntimeError):
    def __init__(self, fn: str, status: int, text: str):
        super().__init__(f"{fn} returned {status}: {text}")
        self.status = status


_vp = ctypes.c_void_p
_SIGNATURES = {
    "moe_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "moe_abi_version": (ctypes.c_int, []),
    "moe_gate_topk": (ctypes.c_int, [_vp, _vp, MoeDims, _vp, _vp, _vp, _vp]),
    "moe_bucket": (ctypes.c_int, [_vp, MoeDims, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "moe_ffn_workspace_bytes": (ctypes.c_size_t, [MoeDims]),
    "moe_expert_ffn": (ctypes.c_int, [_vp] * 7 + [MoeDims, _vp, _vp, ctypes.c_size_t, _vp]),
    "moe_expert_ffn_up": (ctypes.c_int, [_vp] * 6 + [MoeDims, _vp, ctypes.c_size_t, _vp]),
    "moe_expert_ffn_noalloc": (ctypes.c_int, [_vp] * 7 + [MoeDims, _vp, _vp]),
    "moe_expert_ffn_noalloc_max_bytes": (ctypes.c_size_t, []),
    "moe_expert_ffn_up_routed": (ctypes.c_int, [_vp] * 3 + [MoeDims] + [_vp] * 7 +
                                 [ctypes.c_size_t, _vp]),
    "moe_expert_ffn_mxfp4_up_routed": (ctypes.c_int, [_vp] * 4 + [MoeDims] + [_vp] * 7 +
                                       [ctypes.c_size_t, _vp]),
    "moe_expert_ffn_routed": (ctypes.c_int, [_vp] * 4 + [MoeDims] + [_vp] * 8 +
                              [ctypes.c_size_t, _vp, _vp]),
    "moe_expert_ffn_mxfp4_routed": (ctypes.c_int, [_vp] * 6 + [MoeDims] + [_vp] * 8 +
                                    [ctypes.c_size_t, _vp, _vp]),
    "moe_ffn_sync_bytes": (ctypes.c_size_t, [MoeDims]),
    "moe_expert_ffn_down": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _vp, MoeDims, ctypes.c_size_t,
                                           _vp, _vp]),
    "moe_combine": (ctypes.c_int, [_vp, _vp, _vp, MoeDims, _vp, _vp]),
    "moe_pack_up_weights": (ctypes.c_int, [_vp, _vp] + [ctypes.c_int32] * 3 + [_vp, _vp]),
    "moe_pack_down_weights": (ctypes.c_int, [_vp] + [ctypes.c_int32] * 3 + [_vp, _vp]),
    "moe_pack_mxfp4_up": (ctypes.c_int, [_vp, _vp, _vp, _vp, ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int32, _vp, _vp, _vp]),
    "moe_pack_mxfp4_down": (ctypes.c_int, [_vp, _vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           _vp, _vp, _vp]),
    "moe_expert_ffn_mxfp4": (ctypes.c_int, [_vp] * 9 + [MoeDims, _vp, _vp, ctypes.c_size_t, _vp]),
    "moe_expert_ffn_mxfp4_up": (ctypes.c_int, [_vp] * 7 + [MoeDims, _vp, ctypes.c_size_t, _vp]),
    "moe_expert_ffn_mxfp4_down": (ctypes.c_int, [_vp] * 7 + [MoeDims, ctypes.c_size_t, _vp, _vp]),
    "moe_sig_capture": (ctypes.c_int, [_vp, _vp] + [ctypes.c_int32] * 7 + [_vp, _vp, _vp]),
    "moe_sig_reset": (ctypes.c_int, [_vp] + [ctypes.c_int32] * 4 + [_vp, _vp]),
    "moe_sig_request_counts": (ctypes.c_int, [_vp, _vp, _vp] + [ctypes.c_int32] * 5 + [_vp, _vp]),
    "moe_stream_read_probe": (ctypes.c_int, [_vp, ctypes.c_size_t, _vp, _vp]),
    "eldr_idf": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp]),
    "eldr_signature": (ctypes.c_int, [_vp, _vp, ctypes.c_int32, ctypes.c_int32, _vp,
                                      ctypes.c_int32, _vp]),
    "eldr_rho": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int32, _vp, ctypes.c_int32, _vp,
                                ctypes.c_int32, _vp]),
    "eldr_greedy_layers": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _vp,
                                          _vp, ctypes.c_int32, _vp, ctypes.c_int32, _vp, _vp, _vp]),
    "eldr_balanced_kmeans": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                            _vp, ctypes.c_int32, _vp, _vp, _vp]),
    "eldr_route": (ctypes.c_int, [_vp, ctypes.c_int32, _vp, ctypes.c_int32, _vp, ctypes.c_float,
                                  _vp]),
    "eldr_route_batch": (ctypes.c_int, [_vp, ctypes.c_int32, ctypes.c_int32, _vp, ctypes.c_int32,
                                        _vp, ctypes.c_float, _vp]),
}

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (once); raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2607_00466_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def header_functions(paths=HEADER_PATHS) -> list[str]:
    """Names of the functions the headers under include/ declare."""
    text = "\n".join(open(p).read() for p in paths)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?((?:moe|eldr)_\w+)\s*\(", text,
                                 re.M)))


def status_string(status: int) -> str:
    return load().moe_status_string(status).decode()


def _check(fn: str, status: int) -> None:
    if status != MOE_OK:
        raise MoeError(fn, status, status_string(status))


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, numel: int) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name}: must be a device tensor, got {t.device}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name}: needs at least {numel} elements, has {t.numel()}")


def dims(T: int, H: int, E: int, K: int, I: int) -> MoeDims:
    return MoeDims(T, H, E, K, I)


# ----------------------------------------------------------------------------- entry points

def moe_gate_topk(x, w_gate, d: MoeDims, logits, topk_ids, topk_w, stream=None) -> None:
    _need(x, "x", torch.float32, d.T * d.H)
    _need(w_gate, "w_gate", torch.float32, d.E * d.H)
    _need(logits, "logits", torch.float32, d.T * d.E)
    _need(topk_ids, "topk_ids", torch.int32, d.T * d.K)
    _need(topk_w, "topk_w", torch.float32, d.T * d.K)
    _check("moe_gate_topk", load().moe_gate_topk(_ptr(x), _ptr(w_gate), d, _ptr(logits),
                                                 _ptr(topk_ids), _ptr(topk_w), _stream(stream)))


def moe_bucket(topk_ids, d: MoeDims, counts, offsets, perm_token, pair_pos, union_ids, union_size,
               stream=None) -> None:
    _need(topk_ids, "topk_ids", torch.int32, d.T * d.K)
    _need(counts, "counts", torch.int32, d.E)
    _need(offsets, "offsets", torch.int32, d.E + 1)
    _need(perm_token, "perm_token", torch.int32, d.T * d.K)
    _need(pair_pos, "pair_pos", torch.int32, d.T * d.K)
    _need(union_ids, "union_ids", torch.int32, 2 * d.E)
    _need(union_size, "union_size", torch.int32, 1)
    _check("moe_bucket", load().moe_bucket(_ptr(topk_ids), d, _ptr(counts), _ptr(offsets),
                                           _ptr(perm_token), _ptr(pair_pos), _ptr(union_ids),
                                           _ptr(union_size), _stream(stream)))


def moe_ffn_workspace_bytes(d: MoeDims) -> int:
    return int(load().moe_ffn_workspace_bytes(d))


def moe_expert_ffn(x, w13, w2, offsets, perm_token, union_ids, union_size, d: MoeDims, y_perm,
                   ws, stream=None) -> None:
    """The expert FFN of the union; w13 and w2 as packed by ``pack_expert_weights``."""
    _need(x, "x", torch.float32, d.T * d.H)
    _need(w13, "w13", torch.bfloat16, 2 * d.E * d.I * d.H)
    _need(w2, "w2", torch.bfloat16, d.E * d.H * d.I)
    _need(offsets, "offsets", torch.int32, d.E + 1)
    _need(perm_token, "perm_token", torch.int32, d.T * d.K)
    _need(union_ids, "union_ids", torch.int32, 2 * d.E)
    _need(union_size, "union_size", torch.int32, 1)
    _need(y_perm, "y_perm", torch.float32, d.T * d.K * d.H)
    ws_bytes = _need_ws(ws, d)
    _check("moe_expert_ffn", load().moe_expert_ffn(
        _ptr(x), _ptr(w13), _ptr(w2), _ptr(offsets), _ptr(perm_token), _ptr(union_ids),
        _ptr(union_size), d, _ptr(y_perm), _ptr(ws), ws_bytes, _stream(stream)))


def _need_ws(ws, d: MoeDims) -> int:
    if ws.device.type != "cuda" or not ws.is_contiguous():
        raise ValueError("ws: must be a contiguous device tensor")
    return ws.numel() * ws.element_size()


def moe_expert_ffn_up(x, w13, offsets, perm_token, union_ids, union_size, d: MoeDims, ws,
                      stream=None) -> None:
    _need(x, "x", torch.float32, d.T * d.H)
    _need(w13, "w13", torch.bfloat16, 2 * d.E * d.I * d.H)
    _need_routing(offsets, perm_token, union_ids, union_size, d)
    ws_bytes = _need_ws(ws, d)
    _check("moe_expert_ffn_up", load().moe_expert_ffn_up(
        _ptr(x), _ptr(w13), _ptr(offsets), _ptr(perm_token), _ptr(union_ids),
        _ptr(union_size), d, _ptr(ws), ws_bytes, _stream(stream)))


def _need_buckets(d: MoeDims, counts, offsets, perm_token, pair_pos, union_ids, union_size):
    _need(counts, "counts", torch.int32, d.E)
    _need(offsets, "offsets", torch.int32, d.E + 1)
    _need(perm_token, "perm_token", torch.int32, d.T * d.K)
    _need(pair_pos, "pair_pos", torch.int32, d.T * d.K)
    _need(union_ids, "union_ids", torch.int32, 2 * d.E)
    _need(union_size, "union_size", torch.int32, 1)


def moe_expert_ffn_noalloc(x, w13, w2, offsets, perm_token, union_ids, union_size, d: MoeDims,
                           y_perm, stream=None) -> None:
    """moe_expert_ffn with the library's fixed device workspace (no caller buffer)."""
    _need(x, "x", torch.float32, d.T * d.H)
    _need(w13, "w13", torch.bfloat16, 2 * d.E * d.I * d.H)
    _need(w2, "w2", torch.bfloat16, d.E * d.H * d.I)
    _need(y_perm, "y_perm", torch.float32, d.T * d.K * d.H)
    _need_routing(offsets, perm_token, union_ids, union_size, d)
    _check("moe_expert_ffn_noalloc", load().moe_expert_ffn_noalloc(
        _ptr(x), _ptr(w13), _ptr(w2), _ptr(offsets), _ptr(perm_token), _ptr(union_ids),
        _ptr(union_size), d, _ptr(y_perm), _stream(stream)))


def moe_expert_ffn_up_routed(x, w13, topk_ids, d: MoeDims, counts, offsets, perm_token, pair_pos,
                             union_ids, union_size, ws, stream=None) -> None:
    """moe_bucket then moe_expert_ffn_up, one launch for T <= 64."""
    _need(x, "x", torch.float32, d.T * d.H)
    _need(w13, "w13", torch.bfloat16, 2 * d.E * d.I * d.H)
    _need(topk_ids, "topk_ids", torch.int32, d.T * d.K)
    _need_buckets(d, counts, offsets, perm_token, pair_pos, union_ids, union_size)
    ws_bytes = _need_ws(ws, d)
    _check("moe_expert_ffn_up_routed", load().moe_expert_ffn_up_routed(
        _ptr(x), _ptr(w13), _ptr(topk_ids), d, _ptr(counts), _ptr(offsets), _ptr(perm_token),
        _ptr(pair_pos), _ptr(union_ids), _ptr(union_size), _ptr(ws), ws_bytes, _stream(stream)))


def moe_ffn_sync_bytes(d: MoeDims) -> int:
    return int(load().moe_ffn_sync_bytes(d))


def _need_sync(sync, d: MoeDims) -> None:
    _need(sync, "sync", torch.int32, moe_ffn_sync_bytes(d) // 4)


def moe_expert_ffn_routed(x, w13, w2, topk_ids, d: MoeDims, counts, offsets, perm_token, pair_pos,
                          union_ids, union_size, y_perm, ws, sync, stream=None) -> None:
    """moe_bucket then moe_expert_ffn, one launch for T <= 64.  ``sync`` is an
    int32 [64 E + 1] device tensor (moe_ffn_sync_bytes), zero before the first
    call (left zero)."""
    _need(x, "x", torch.float32, d.T * d.H)
    _need(w13, "w13", torch.bfloat16, 2 * d.E * d.I * d.H)
    _need(w2, "w2", torch.bfloat16, d.E * d.H * d.I)
    _need(topk_ids, "topk_ids", torch.int32, d.T * d.K)
    _need_buckets(d, counts, offsets, perm_token, pair_pos, union_ids, union_size)
    _need(y_perm, "y_perm", torch.float32, d.T * d.K * d.H)
    ws_bytes = _need_ws(ws, d)
    _need_sync(sync, d)
    _check("moe_expert_ffn_routed", load().moe_expert_ffn_routed(
        _ptr(x), _ptr(w13), _ptr(w2), _ptr(topk_ids), d, _ptr(counts), _ptr(offsets),
        _ptr(perm_token), _ptr(pair_pos), _ptr(union_ids), _ptr(union_size), _ptr(y_perm),
        _ptr(ws), ws_bytes, _ptr(sync), _stream(stream)))


def moe_expert_ffn_down(ws, w2, offsets, perm_token, union_ids, union_size, d: MoeDims, y_perm,
                        stream=None) -> None:
    _need(w2, "w2", torch.bfloat16, d.E * d.H * d.I)
    _need(y_perm, "y_perm", torch.float32, d.T * d.K * d.H)
    _need_routing(offsets, perm_token, union_ids, union_size, d)
    ws_bytes = _need_ws(ws, d)
    _check("moe_expert_ffn_down", load().moe_expert_ffn_down(
        _ptr(ws), _ptr(w2), _ptr(offsets), _ptr(perm_token), _ptr(union_ids), _ptr(union_size), d,
        ws_bytes, _ptr(y_perm), _stream(stream)))


def moe_pack_up_weights(w1, w3, dst=None, stream=None) -> torch.Tensor:
    """Pack W1 and W3 ([E, I, H] bf16 each) into one band-interleaved tensor; returns dst."""
    if w1.dim() != 3 or w1.shape != w3.shape:
        raise ValueError("w1, w3: expected two [E, I, H] tensors")
    E, I, H = (int(v) for v in w1.shape)
    _need(w1, "w1", torch.bfloat16, E * I * H)
    _need(w3, "w3", torch.bfloat16, E * I * H)
    if dst is None:
        dst = torch.empty((E, 2 * I, H), dtype=torch.bfloat16, device=w1.device)
    _need(dst, "dst", torch.bfloat16, 2 * E * I * H)
    _check("moe_pack_up_weights", load().moe_pack_up_weights(_ptr(w1), _ptr(w3), E, I, H, _ptr(dst),
                                                             _stream(stream)))
    return dst


def moe_pack_down_weights(w2, dst=None, stream=None) -> torch.Tensor:
    """Pack W2 ([E, H, I] bf16) band by band for the down projection; returns dst."""
    if w2.dim() != 3:
        raise ValueError("w2: expected [E, H, I]")
    E, H, I = (int(v) for v in w2.shape)
    _need(w2, "w2", torch.bfloat16, E * H * I)
    if dst is None:
        dst = torch.empty_like(w2)
    _need(dst, "dst", torch.bfloat16, E * H * I)
    _check("moe_pack_down_weights", load().moe_pack_down_weights(_ptr(w2), E, H, I, _ptr(dst),
                                                                 _stream(stream)))
    return dst


def pack_expert_weights(w1, w3, w2, stream=None):
    """Pack (w1 [E,I,H], w3 [E,I,H], w2 [E,H,I]) for moe_expert_ffn: returns (w13, w2p)."""
    return (moe_pack_up_weights(w1, w3, stream=stream), moe_pack_down_weights(w2, stream=stream))


# ----------------------------------------------------------------------------- MXFP4 experts
#
# An MXFP4 weight is a pair (codes, scales) of uint8 device tensors: codes
# [E, R, K/2] (two E2M1 codes a byte, the even index in the low nibble) and
# scales [E, R, K/32] (E8M0), as checkpoints store them; packed pairs are
# flat uint8 tensors of the same sizes.

def _need_u8(t, name: str, numel: int) -> None:
    _need(t, name, torch.uint8, numel)


def moe_pack_mxfp4_up(w1, w3, stream=None):
    """Pack W1 and W3 (each (codes [E,I,H/2], scales [E,I,H/32])); returns (codes, scales)."""
    (c1, s1), (c3, s3) = w1, w3
    if c1.dim() != 3:
        raise ValueError("codes: expected [E, R, K/2]")
    E, I, H = int(c1.shape[0]), int(c1.shape[1]), int(c1.shape[2]) * 2
    for name, t, n in (("w1 codes", c1, E * I * H // 2), ("w3 codes", c3, E * I * H // 2),
                       ("w1 scales", s1, E * I * H // 32), ("w3 scales", s3, E * I * H // 32)):
        _need_u8(t, name, n)
    codes = torch.empty(E * I * H, dtype=torch.uint8, device=c1.device)
    scales = torch.empty(E * I * H // 16, dtype=torch.uint8, device=c1.device)
    _check("moe_pack_mxfp4_up", load().moe_pack_mxfp4_up(
        _ptr(c1), _ptr(s1), _ptr(c3), _ptr(s3), E, I, H, _ptr(codes), _ptr(scales), _stream(stream)))
    return codes, scales


def moe_pack_mxfp4_down(w2, stream=None):
    """Pack W2 ((codes [E,H,I/2], scales [E,H,I/32])); returns (codes, scales)."""
    c2, s2 = w2
    if c2.dim() != 3:
        raise ValueError("codes: expected [E, R, K/2]")
    E, H, I = int(c2.shape[0]), int(c2.shape[1]), int(c2.shape[2]) * 2
    _need_u8(c2, "w2 codes", E * H * I // 2)
    _need_u8(s2, "w2 scales", E * H * I // 32)
    codes = torch.empty(E * H * I // 2, dtype=torch.uint8, device=c2.device)
    scales = torch.empty(E * H * I // 32, dtype=torch.uint8, device=c2.device)
    _check("moe_pack_mxfp4_down", load().moe_pack_mxfp4_down(
        _ptr(c2), _ptr(s2), E, H, I, _ptr(codes), _ptr(scales), _stream(stream)))
    return codes, scales


def pack_mxfp4_expert_weights(w1, w3, w2, stream=None):
    """Pack MXFP4 (w1, w3, w2) for moe_expert_ffn_mxfp4; returns (up, down) pairs."""
    return moe_pack_mxfp4_up(w1, w3, stream), moe_pack_mxfp4_down(w2, stream)


def _need_mx_up(up, d: MoeDims) -> None:
    _need_u8(up[0], "up codes", d.E * d.I * d.H)
    _need_u8(up[1], "up scales", d.E * d.I * d.H // 16)


def _need_mx_down(down, d: MoeDims) -> None:
    _need_u8(down[0], "down codes", d.E * d.H * d.I // 2)
    _need_u8(down[1], "down scales", d.E * d.H * d.I // 32)


def _need_routing(offsets, perm_token, union_ids, union_size, d: MoeDims) -> None:
    _need(offsets, "offsets", torch.int32, d.E + 1)
    _need(perm_token, "perm_token", torch.int32, d.T * d.K)
    _need(union_ids, "union_ids", torch.int32, 2 * d.E)
    _need(union_size, "union_size", torch.int32, 1)


def moe_expert_ffn_mxfp4(x, up, down, offsets, perm_token, union_ids, union_size, d: MoeDims,
                         y_perm, ws, stream=None) -> None:
    _need(x, "x", torch.float32, d.T * d.H)
    _need_mx_up(up, d)
    _need_mx_down(down, d)
    _need_routing(offsets, perm_token, union_ids, union_size, d)
    _need(y_perm, "y_perm", torch.float32, d.T * d.K * d.H)
    ws_bytes = _need_ws(ws, d)
    _check("moe_expert_ffn_mxfp4", load().moe_expert_ffn_mxfp4(
        _ptr(x), _ptr(up[0]), _ptr(up[1]), _ptr(down[0]), _ptr(down[1]), _ptr(offsets),
        _ptr(perm_token), _ptr(union_ids), _ptr(union_size), d, _ptr(y_perm), _ptr(ws), ws_bytes,
        _stream(stream)))


def moe_expert_ffn_mxfp4_up(x, up, offsets, perm_token, union_ids, union_size, d: MoeDims, ws,
                            stream=None) -> None:
    _need(x, "x", torch.float32, d.T * d.H)
    _need_mx_up(up, d)
    _need_routing(offsets, perm_token, union_ids, union_size, d)
    ws_bytes = _need_ws(ws, d)
    _check("moe_expert_ffn_mxfp4_up", load().moe_expert_ffn_mxfp4_up(
        _ptr(x), _ptr(up[0]), _ptr(up[1]), _ptr(offsets), _ptr(perm_token), _ptr(union_ids),
        _ptr(union_size), d, _ptr(ws), ws_bytes, _stream(stream)))


def moe_expert_ffn_mxfp4_up_routed(x, up, topk_ids, d: MoeDims, counts, offsets, perm_token,
                                   pair_pos, union_ids, union_size, ws, stream=None) -> None:
    """moe_bucket then moe_expert_ffn_mxfp4_up, one launch for T <= 64."""
    _need(x, "x", torch.float32, d.T * d.H)
    _need_mx_up(up, d)
    _need(topk_ids, "topk_ids", torch.int32, d.T * d.K)
    _need_buckets(d, counts, offsets, perm_token, pair_pos, union_ids, union_size)
    ws_bytes = _need_ws(ws, d)
    _check("moe_expert_ffn_mxfp4_up_routed", load().moe_expert_ffn_mxfp4_up_routed(
        _ptr(x), _ptr(up[0]), _ptr(up[1]), _ptr(topk_ids), d, _ptr(counts), _ptr(offsets),
        _ptr(perm_token), _ptr(pair_pos), _ptr(union_ids), _ptr(union_size), _ptr(ws), ws_bytes,
        _stream(stream)))


def moe_expert_ffn_mxfp4_routed(x, up, down, topk_ids, d: MoeDims, counts, offsets, perm_token,
                                pair_pos, union_ids, union_size, y_perm, ws, sync,
                                stream=None) -> None:
    """moe_bucket then moe_expert_ffn_mxfp4, one launch for T <= 64 (``sync`` as
    for moe_expert_ffn_routed)."""
    _need(x, "x", torch.float32, d.T * d.H)
    _need_mx_up(up, d)
    _need_mx_down(down, d)
    _need(topk_ids, "topk_ids", torch.int32, d.T * d.K)
    _need_buckets(d, counts, offsets, perm_token, pair_pos, union_ids, union_size)
    _need(y_perm, "y_perm", torch.float32, d.T * d.K * d.H)
    ws_bytes = _need_ws(ws, d)
    _need_sync(sync, d)
    _check("moe_expert_ffn_mxfp4_routed", load().moe_expert_ffn_mxfp4_routed(
        _ptr(x), _ptr(up[0]), _ptr(up[1]), _ptr(down[0]), _ptr(down[1]), _ptr(topk_ids), d,
        _ptr(counts), _ptr(offsets), _ptr(perm_token), _ptr(pair_pos), _ptr(union_ids),
        _ptr(union_size), _ptr(y_perm), _ptr(ws), ws_bytes, _ptr(sync), _stream(stream)))


def moe_expert_ffn_mxfp4_down(ws, down, offsets, perm_token, union_ids, union_size, d: MoeDims,
                              y_perm, stream=None) -> None:
    _need_mx_down(down, d)
    _need_routing(offsets, perm_token, union_ids, union_size, d)
    _need(y_perm, "y_perm", torch.float32, d.T * d.K * d.H)
    ws_bytes = _need_ws(ws, d)
    _check("moe_expert_ffn_mxfp4_down", load().moe_expert_ffn_mxfp4_down(
        _ptr(ws), _ptr(down[0]), _ptr(down[1]), _ptr(offsets), _ptr(perm_token), _ptr(union_ids),
        _ptr(union_size), d, ws_bytes, _ptr(y_perm), _stream(stream)))


def moe_combine(y_perm, pair_pos, topk_w, d: MoeDims, out, stream=None) -> None:
    _need(y_perm, "y_perm", torch.float32, d.T * d.K * d.H)
    _need(pair_pos, "pair_pos", torch.int32, d.T * d.K)
    _need(topk_w, "topk_w", torch.float32, d.T * d.K)
    _need(out, "out", torch.float32, d.T * d.H)
    _check("moe_combine", load().moe_combine(_ptr(y_perm), _ptr(pair_pos), _ptr(topk_w), d,
                                             _ptr(out), _stream(stream)))


# ----------------------------------------------------------------------------- a whole layer

@dataclass
class LayerBuffers:
    """Device buffers of one layer invocation (allocated once, reused every step)."""

    logits: torch.Tensor
    topk_ids: torch.Tensor
    topk_w: torch.Tensor
    counts: torch.Tensor
    offsets: torch.Tensor
    perm_token: torch.Tensor
    pair_pos: torch.Tensor
    union_ids: torch.Tensor
    union_size: torch.Tensor
    y_perm: torch.Tensor
    ws: torch.Tensor
    out: torch.Tensor
    sync: torch.Tensor  # moe_expert_ffn_routed's counters: zero at allocation, left zero by every call

    @classmethod
    def allocate(cls, d: MoeDims, device="cuda") -> "LayerBuffers":
        i32 = dict(dtype=torch.int32, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        nbytes = moe_ffn_workspace_bytes(d)
        return cls(
            logits=torch.empty((d.T, d.E), **f32),
            topk_ids=torch.empty((d.T, d.K), **i32),
            topk_w=torch.empty((d.T, d.K), **f32),
            counts=torch.empty(d.E, **i32),
            offsets=torch.empty(d.E + 1, **i32),
            perm_token=torch.empty(max(1, d.T * d.K), **i32),
            pair_pos=torch.empty(max(1, d.T * d.K), **i32),
            union_ids=torch.empty(2 * d.E, **i32),
            union_size=torch.empty(1, **i32),
            y_perm=torch.empty((max(1, d.T * d.K), d.H), **f32),
            ws=torch.empty(max(16, nbytes) // 4, **f32),
            out=torch.empty((d.T, d.H), **f32),
            sync=torch.zeros(max(1, moe_ffn_sync_bytes(d) // 4), **i32),
        )


def _gate(x, w_gate, d: MoeDims, buf: LayerBuffers, routing, stream):
    """The gate (unless routing is given); returns the routing (ids, weights)."""
    if routing is None:
        moe_gate_topk(x, w_gate, d, buf.logits, buf.topk_ids, buf.topk_w, stream)
        return buf.topk_ids, buf.topk_w
    return routing


# How moe_layer and moe_layer_mxfp4 run the expert FFN:
#   "fused":  moe_expert_ffn_routed -- buckets, up and down projections in one launch;
#   "routed": moe_expert_ffn_up_routed (buckets + up), then moe_expert_ffn_down;
#   "split":  moe_bucket, moe_expert_ffn_up, moe_expert_ffn_down.
# All three leave the same buffers, bit for bit.
FFN_PATHS = ("fused", "routed", "split")


def moe_layer(x, w_gate, w13, w2, d: MoeDims, buf: LayerBuffers, routing=None, stream=None,
              path: str = "routed"):
    """One decode-step MoE layer on one stream: gate, buckets and expert FFN
    (buckets + up projection in one launch, then down, by default: see
    FFN_PATHS), combine.

    w13 and w2 are the expert weights packed by ``pack_expert_weights``.

    ``routing=(topk_ids, topk_w)`` (int32 [T, K] and fp32 [T, K] device
    tensors) bypasses the gate: the buckets and the combine read them in place.
    Returns ``buf.out``.
    """
    ids, w = _gate(x, w_gate, d, buf, routing, stream)
    if path == "fused":
        moe_expert_ffn_routed(x, w13, w2, ids, d, buf.counts, buf.offsets, buf.perm_token,
                              buf.pair_pos, buf.union_ids, buf.union_size, buf.y_perm, buf.ws,
                              buf.sync, stream)
    elif path in ("routed", "split"):
        if path == "routed":
            moe_expert_ffn_up_routed(x, w13, ids, d, buf.counts, buf.offsets, buf.perm_token,
                                     buf.pair_pos, buf.union_ids, buf.union_size, buf.ws, stream)
        else:
            moe_bucket(ids, d, buf.counts, buf.offsets, buf.perm_token, buf.pair_pos,
                       buf.union_ids, buf.union_size, stream)
            moe_expert_ffn_up(x, w13, buf.offsets, buf.perm_token, buf.union_ids, buf.union_size,
                              d, buf.ws, stream)
        moe_expert_ffn_down(buf.ws, w2, buf.offsets, buf.perm_token, buf.union_ids,
                            buf.union_size, d, buf.y_perm, stream)
    else:
        raise ValueError(f"unknown FFN path {path!r} (one of {FFN_PATHS})")
    moe_combine(buf.y_perm, buf.pair_pos, w, d, buf.out, stream)
    return buf.out


def moe_layer_mxfp4(x, w_gate, up, down, d: MoeDims, buf: LayerBuffers, routing=None, stream=None,
                    path: str = "routed"):
    """moe_layer with MXFP4 experts: ``up`` and ``down`` from pack_mxfp4_expert_weights."""
    ids, w = _gate(x, w_gate, d, buf, routing, stream)
    if path == "fused":
        moe_expert_ffn_mxfp4_routed(x, up, down, ids, d, buf.counts, buf.offsets, buf.perm_token,
                                    buf.pair_pos, buf.union_ids, buf.union_size, buf.y_perm,
                                    buf.ws, buf.sync, stream)
    elif path in ("routed", "split"):
        if path == "routed":
            moe_expert_ffn_mxfp4_up_routed(x, up, ids, d, buf.counts, buf.offsets, buf.perm_token,
                                           buf.pair_pos, buf.union_ids, buf.union_size, buf.ws,
                                           stream)
        else:
            moe_bucket(ids, d, buf.counts, buf.offsets, buf.perm_token, buf.pair_pos,
                       buf.union_ids, buf.union_size, stream)
            moe_expert_ffn_mxfp4_up(x, up, buf.offsets, buf.perm_token, buf.union_ids,
                                    buf.union_size, d, buf.ws, stream)
        moe_expert_ffn_mxfp4_down(buf.ws, down, buf.offsets, buf.perm_token, buf.union_ids,
                                  buf.union_size, d, buf.y_perm, stream)
    else:
        raise ValueError(f"unknown FFN path {path!r} (one of {FFN_PATHS})")
    moe_combine(buf.y_perm, buf.pair_pos, w, d, buf.out, stream)
    return buf.out


# ----------------------------------------------------------------------------- signature cache

def moe_sig_capture(ids, token_block, layer0: int, L: int, E: int, sig, rejected=None,
                    stream=None) -> None:
    """Add one forward's picks ids [n_layers, T, K] to the int8 cache sig [num_blocks, L, E]."""
    if ids.dim() != 3:
        raise ValueError("ids: expected [n_layers, T, K]")
    n_layers, T, K = ids.shape
    if sig.dim() != 3 or tuple(sig.shape[1:]) != (L, E):
        raise ValueError("sig: expected [num_blocks, L, E]")
    _need(ids, "ids", torch.int32, n_layers * T * K)
    _need(token_block, "token_block", torch.int32, T)
    _need(sig, "sig", torch.int8, sig.numel())
    if rejected is not None:
        _need(rejected, "rejected", torch.int32, 1)
    _check("moe_sig_capture", load().moe_sig_capture(
        _ptr(ids), _ptr(token_block), n_layers, T, K, layer0, L, E, sig.shape[0], _ptr(sig),
        _ptr(rejected), _stream(stream)))


def moe_sig_reset(blocks, sig, stream=None) -> None:
    """Zero the rows of the listed blocks of sig [num_blocks, L, E]."""
    _need(blocks, "blocks", torch.int32, blocks.numel())
    _need(sig, "sig", torch.int8, sig.numel())
    nb, L, E = sig.shape
    _check("moe_sig_reset", load().moe_sig_reset(_ptr(blocks), blocks.numel(), L, E, nb, _ptr(sig),
                                                 _stream(stream)))


def moe_sig_request_counts(sig, block_table, n_blocks, out=None, stream=None) -> torch.Tensor:
    """Per-request sums of block rows: out [R, L, E] int32."""
    nb, L, E = sig.shape
    R, max_blocks = block_table.shape
    _need(sig, "sig", torch.int8, sig.numel())
    _need(block_table, "block_table", torch.int32, R * max_blocks)
    _need(n_blocks, "n_blocks", torch.int32, R)
    if out is None:
        out = torch.empty((R, L, E), dtype=torch.int32, device=sig.device)
    _need(out, "out", torch.int32, R * L * E)
    _check("moe_sig_request_counts", load().moe_sig_request_counts(
        _ptr(sig), _ptr(block_table), _ptr(n_blocks), R, max_blocks, L, E, nb, _ptr(out),
        _stream(stream)))
    return out


# ----------------------------------------------------------------------------- calibration

def moe_stream_read_probe(buf, sink, stream=None) -> None:
    """Read all of buf once with the plain streaming kernel (measurement aid)."""
    if buf.device.type != "cuda" or not buf.is_contiguous():
        raise ValueError("buf: must be a contiguous device tensor")
    _need(sink, "sink", torch.int32, 1)
    _check("moe_stream_read_probe", load().moe_stream_read_probe(
        _ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), _stream(stream)))


# ----------------------------------------------------------------------------- routing (host)

def _host(a, dtype):
    """A C-contiguous NumPy array of `dtype` and a pointer to it (host memory)."""
    import numpy as np

    arr = np.ascontiguousarray(a, dtype=dtype)
    return arr, ctypes.c_void_p(arr.ctypes.data)


def eldr_idf(counts):
    """IDF table [L, E] float32 from calibration counts [N, L, E]."""
    import numpy as np

    c, pc = _host(counts, np.int32)
    N, L, E = c.shape
    out = np.empty((L, E), np.float32)
    _check("eldr_idf", load().eldr_idf(pc, N, L, E, ctypes.c_void_p(out.ctypes.data)))
    return out


def eldr_signature(counts, idf, layers):
    """Signature [len(layers) * E] float32 of one request's counts [L, E]."""
    import numpy as np

    c, pc = _host(counts, np.int32)
    w, pw = _host(idf, np.float32)
    ly, pl = _host(layers, np.int32)
    L, E = c.shape
    out = np.empty(len(ly) * E, np.float32)
    _check("eldr_signature", load().eldr_signature(pc, pw, L, E, pl, len(ly),
                                                   ctypes.c_void_p(out.ctypes.data)))
    return out


def eldr_rho(S, P, pairs) -> float:
    import numpy as np

    s, ps = _host(S, np.float32)
    p, pp = _host(P, np.float32)
    pr, ppr = _host(pairs, np.int32)
    out = ctypes.c_double(0.0)
    _check("eldr_rho", load().eldr_rho(ps, s.shape[0], s.shape[1], pp, p.shape[1], ppr, pr.shape[0],
                                       ctypes.byref(out)))
    return out.value


def eldr_greedy_layers(counts, idf, P, pairs):
    """(order [L], rho curve [L], N*) of greedy layer selection."""
    import numpy as np

    c, pc = _host(counts, np.int32)
    w, pw = _host(idf, np.float32)
    p, pp = _host(P, np.float32)
    pr, ppr = _host(pairs, np.int32)
    N, L, E = c.shape
    order = np.empty(L, np.int32)
    curve = np.empty(L, np.float64)
    n_star = ctypes.c_int32(0)
    _check("eldr_greedy_layers", load().eldr_greedy_layers(
        pc, N, L, E, pw, pp, p.shape[1], ppr, pr.shape[0], ctypes.c_void_p(order.ctypes.data),
        ctypes.c_void_p(curve.ctypes.data), ctypes.byref(n_star)))
    return order, curve, n_star.value


def eldr_balanced_kmeans(S, K: int, init, max_iters: int = 50):
    """(centroids [K, d] float32, assignment [N] int32, iterations) of balanced K-means."""
    import numpy as np

    s, ps = _host(S, np.float32)
    ini, pi = _host(init, np.int32)
    N, d = s.shape
    C = np.empty((K, d), np.float32)
    assign = np.empty(N, np.int32)
    iters = ctypes.c_int32(0)
    _check("eldr_balanced_kmeans", load().eldr_balanced_kmeans(
        ps, N, d, K, pi, max_iters, ctypes.c_void_p(C.ctypes.data),
        ctypes.c_void_p(assign.ctypes.data), ctypes.byref(iters)))
    return C, assign, iters.value


def eldr_route(s, centroids, loads, tau: float) -> int:
    import numpy as np

    v, pv = _host(s, np.float32)
    c, pc = _host(centroids, np.float32)
    ld, pld = _host(loads, np.int32)
    out = ctypes.c_int32(-1)
    _check("eldr_route", load().eldr_route(pv, v.shape[0], pc, c.shape[0], pld, tau,
                                           ctypes.byref(out)))
    return out.value


def eldr_route_batch(S, centroids, loads, tau: float):
    """Route the rows of S in order; returns (workers [R], loads after routing [K])."""
    import numpy as np

    s, ps = _host(S, np.float32)
    c, pc = _host(centroids, np.float32)
    ld = np.array(loads, dtype=np.int32, copy=True)
    workers = np.empty(s.shape[0], np.int32)
    _check("eldr_route_batch", load().eldr_route_batch(
        ps, s.shape[0], s.shape[1], pc, c.shape[0], ctypes.c_void_p(ld.ctypes.data), tau,
        ctypes.c_void_p(workers.ctypes.data)))
    return workers, ld
