"""The C-ABI library loads, exports what its header declares, and rejects bad
arguments on the host before anything is launched (no GPU needed)."""
import ctypes
import re

import pytest

from paper_2607_00466_amd import binding as B

FAKE = ctypes.c_void_p(0x10000)        # 16-byte aligned, never dereferenced
FAKE_MIS = ctypes.c_void_p(0x10004)    # 4-byte aligned only


@pytest.fixture(scope="module")
def lib():
    return B.load()


def test_exports_every_declared_function(lib):
    names = B.header_functions()
    assert {"moe_gate_topk", "moe_bucket", "moe_expert_ffn", "moe_expert_ffn_up",
            "moe_expert_ffn_down", "moe_combine", "moe_pack_up_weights", "moe_pack_down_weights",
            "moe_ffn_workspace_bytes", "moe_status_string", "moe_abi_version",
            "moe_sig_capture", "moe_sig_reset", "moe_sig_request_counts",
            "moe_stream_read_probe"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    assert lib.moe_abi_version() == 2
    for st in (B.MOE_OK, B.MOE_ERR_INVALID, B.MOE_ERR_UNSUPPORTED, B.MOE_ERR_WORKSPACE, B.MOE_ERR_HIP):
        assert B.status_string(st).startswith("MOE_")
    assert B.status_string(12345) == "unknown status"


def test_limits_match_the_header():
    text = open(B.HEADER_PATH).read()
    for name in ("MOE_MAX_E", "MOE_MAX_K", "MOE_MAX_T", "MOE_MAX_H", "MOE_MAX_I"):
        m = re.search(rf"#define {name} (\d+)", text)
        assert m and int(m.group(1)) == getattr(B, name), name


def test_workspace_bytes(lib):
    assert B.moe_ffn_workspace_bytes(B.dims(64, 2048, 128, 8, 768)) == 4 * 64 * 8 * 768
    assert B.moe_ffn_workspace_bytes(B.dims(0, 2048, 128, 8, 768)) == 0
    assert B.moe_ffn_workspace_bytes(B.dims(8, 2048, 4, 8, 768)) == 0  # K > E is invalid


GOOD = (64, 2048, 128, 8, 768)


@pytest.mark.parametrize("dims,status", [
    ((64, 2048, 128, 129, 768), B.MOE_ERR_INVALID),      # K > E
    ((-1, 2048, 128, 8, 768), B.MOE_ERR_INVALID),        # negative T
    ((64, 0, 128, 8, 768), B.MOE_ERR_INVALID),           # H = 0
    ((64, 2048, 257, 8, 768), B.MOE_ERR_UNSUPPORTED),    # E above the limit
    ((64, 2048, 128, 17, 768), B.MOE_ERR_UNSUPPORTED),   # K above the limit
    ((4097, 2048, 128, 8, 768), B.MOE_ERR_UNSUPPORTED),  # T above the limit
    ((64, 2040, 128, 8, 768), B.MOE_ERR_UNSUPPORTED),    # H not a multiple of 32
    ((64, 2048, 128, 8, 760), B.MOE_ERR_UNSUPPORTED),    # I not a multiple of 32
])
def test_dims_rejected_by_every_call(lib, dims, status):
    d = B.dims(*dims)
    s = None
    assert lib.moe_gate_topk(FAKE, FAKE, d, FAKE, FAKE, FAKE, s) == status
    assert lib.moe_bucket(FAKE, d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, s) == status
    assert lib.moe_expert_ffn(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, d, FAKE, FAKE,
                              1 << 40, s) == status
    assert lib.moe_combine(FAKE, FAKE, FAKE, d, FAKE, s) == status


def test_null_pointers_rejected(lib):
    d = B.dims(*GOOD)
    assert lib.moe_gate_topk(None, FAKE, d, FAKE, FAKE, FAKE, None) == B.MOE_ERR_INVALID
    assert lib.moe_bucket(FAKE, d, None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == B.MOE_ERR_INVALID
    assert lib.moe_expert_ffn(FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, d, FAKE, FAKE,
                              1 << 40, None) == B.MOE_ERR_INVALID
    assert lib.moe_combine(FAKE, FAKE, FAKE, d, None, None) == B.MOE_ERR_INVALID


def test_misaligned_pointers_rejected(lib):
    d = B.dims(*GOOD)
    assert lib.moe_gate_topk(FAKE_MIS, FAKE, d, FAKE, FAKE, FAKE, None) == B.MOE_ERR_UNSUPPORTED
    assert lib.moe_expert_ffn(FAKE, FAKE_MIS, FAKE, FAKE, FAKE, FAKE, FAKE, d, FAKE, FAKE,
                              1 << 40, None) == B.MOE_ERR_UNSUPPORTED
    assert lib.moe_combine(FAKE_MIS, FAKE, FAKE, d, FAKE, None) == B.MOE_ERR_UNSUPPORTED
    odd = ctypes.c_void_p(0x10002)
    assert lib.moe_bucket(odd, d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == B.MOE_ERR_UNSUPPORTED


def test_workspace_too_small_rejected(lib):
    d = B.dims(*GOOD)
    need = B.moe_ffn_workspace_bytes(d)
    assert lib.moe_expert_ffn(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, d, FAKE, FAKE,
                              need - 1, None) == B.MOE_ERR_WORKSPACE


def test_bucket_bitmap_limit(lib):
    # E * ceil(T / 32) must stay within 16384 words of LDS bitmaps.
    d = B.dims(4096, 2048, 256, 8, 768)
    assert lib.moe_bucket(FAKE, d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == B.MOE_ERR_UNSUPPORTED


def test_empty_batch_is_a_no_op(lib):
    # T = 0: gate, ffn and combine return before any launch.
    d = B.dims(0, 2048, 128, 8, 768)
    assert lib.moe_gate_topk(None, None, d, None, None, None, None) == B.MOE_OK
    assert lib.moe_expert_ffn(None, None, None, None, None, None, None, d, None, None, 0,
                              None) == B.MOE_OK
    assert lib.moe_combine(None, None, None, d, None, None) == B.MOE_OK


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    # No CPU fallback: without the built HIP library every call path raises.
    monkeypatch.setattr(B, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        B.load(str(tmp_path / "libeldr_moe.so"))
    assert B._lib is None


def test_binding_requires_device_tensors():
    import torch
    d = B.dims(2, 64, 4, 2, 32)
    with pytest.raises(ValueError):
        B.moe_combine(torch.zeros(4, 64), torch.zeros(4, dtype=torch.int32), torch.zeros(2, 2), d,
                      torch.zeros(2, 64))


def test_pack_arguments_rejected(lib):
    FAKE2 = ctypes.c_void_p(0x20000)
    up, down = lib.moe_pack_up_weights, lib.moe_pack_down_weights
    assert up(FAKE, FAKE, -1, 32, 32, FAKE2, None) == B.MOE_ERR_INVALID
    assert up(FAKE, FAKE, 2, 48, 32, FAKE2, None) == B.MOE_ERR_UNSUPPORTED    # I % 32
    assert up(FAKE, FAKE, 2, 32, 48, FAKE2, None) == B.MOE_ERR_UNSUPPORTED    # H % 32
    assert up(FAKE, None, 2, 32, 32, FAKE2, None) == B.MOE_ERR_INVALID
    assert up(FAKE, FAKE2, 2, 32, 32, FAKE2, None) == B.MOE_ERR_INVALID       # in place
    assert up(FAKE_MIS, FAKE, 2, 32, 32, FAKE2, None) == B.MOE_ERR_UNSUPPORTED
    assert up(None, None, 0, 32, 32, None, None) == B.MOE_OK                  # empty
    assert down(FAKE, 2, 48, 32, FAKE2, None) == B.MOE_ERR_UNSUPPORTED        # H % 32
    assert down(None, 2, 32, 32, FAKE2, None) == B.MOE_ERR_INVALID
    assert down(FAKE, 2, 32, 32, FAKE, None) == B.MOE_ERR_INVALID             # in place
    assert down(None, 2, 32, 0, None, None) == B.MOE_OK                       # empty


def test_signature_calls_validate_on_host(lib):
    # moe_sig_capture(ids, token_block, n_layers, T, K, layer0, L, E, num_blocks, sig, rejected, stream)
    cap = lib.moe_sig_capture
    assert cap(FAKE, FAKE, 1, 64, 8, 0, 3, 7, 10, FAKE, None, None) == B.MOE_ERR_UNSUPPORTED  # L*E % 4
    assert cap(FAKE, FAKE, 4, 64, 8, 45, 48, 128, 10, FAKE, None, None) == B.MOE_ERR_INVALID  # layers past L
    assert cap(FAKE, FAKE, 1, 64, 9, 0, 4, 8, 10, FAKE, None, None) == B.MOE_ERR_INVALID      # K > E
    assert cap(None, FAKE, 1, 64, 8, 0, 4, 128, 10, FAKE, None, None) == B.MOE_ERR_INVALID
    assert cap(FAKE, FAKE, 1, 0, 8, 0, 4, 128, 10, None, None, None) == B.MOE_OK              # nothing to add
    assert cap(FAKE, FAKE, 0, 64, 8, 0, 4, 128, 10, None, None, None) == B.MOE_OK
    odd = ctypes.c_void_p(0x10002)
    assert cap(FAKE, FAKE, 1, 64, 8, 0, 4, 128, 10, odd, None, None) == B.MOE_ERR_UNSUPPORTED
    assert cap(FAKE, FAKE, 1, 64, 8, 0, 4, 512, 10, FAKE, None, None) == B.MOE_ERR_UNSUPPORTED  # E > 256
    # moe_sig_reset(blocks, n, L, E, num_blocks, sig, stream)
    assert lib.moe_sig_reset(FAKE, 0, 4, 128, 10, FAKE, None) == B.MOE_OK
    assert lib.moe_sig_reset(FAKE, -1, 4, 128, 10, FAKE, None) == B.MOE_ERR_INVALID
    assert lib.moe_sig_reset(None, 3, 4, 128, 10, FAKE, None) == B.MOE_ERR_INVALID
    # moe_sig_request_counts(sig, table, n_blocks, R, max_blocks, L, E, num_blocks, out, stream)
    rc = lib.moe_sig_request_counts
    assert rc(FAKE, FAKE, FAKE, 0, 8, 4, 128, 10, FAKE, None) == B.MOE_OK
    assert rc(FAKE, FAKE, FAKE, 3, 8, 4, 128, 10, FAKE_MIS, None) == B.MOE_ERR_UNSUPPORTED  # out needs 16 B
    assert rc(FAKE, FAKE, None, 3, 8, 4, 128, 10, FAKE, None) == B.MOE_ERR_INVALID
    assert rc(FAKE, FAKE, FAKE, -1, 8, 4, 128, 10, FAKE, None) == B.MOE_ERR_INVALID


def test_stream_probe_validates_on_host(lib):
    assert lib.moe_stream_read_probe(FAKE, 0, FAKE, None) == B.MOE_OK
    assert lib.moe_stream_read_probe(None, 64, FAKE, None) == B.MOE_ERR_INVALID
    assert lib.moe_stream_read_probe(FAKE, 24, FAKE, None) == B.MOE_ERR_UNSUPPORTED
    assert lib.moe_stream_read_probe(FAKE_MIS, 64, FAKE, None) == B.MOE_ERR_UNSUPPORTED


def test_mxfp4_calls_validate_on_host(lib):
    ffn, up, down = lib.moe_expert_ffn_mxfp4, lib.moe_expert_ffn_mxfp4_up, lib.moe_expert_ffn_mxfp4_down
    d = B.dims(64, 2880, 128, 4, 2880)
    need = B.moe_ffn_workspace_bytes(d)
    args9 = [FAKE] * 9
    # H or I not a multiple of 64 (the MXFP4 slot), though multiples of 32
    for bad in (B.dims(64, 2880 + 32, 128, 4, 2880), B.dims(64, 2880, 128, 4, 2880 - 32)):
        assert ffn(*args9, bad, FAKE, FAKE, 1 << 40, None) == B.MOE_ERR_UNSUPPORTED
        assert up(*[FAKE] * 7, bad, FAKE, 1 << 40, None) == B.MOE_ERR_UNSUPPORTED
        assert down(*[FAKE] * 7, bad, 1 << 40, FAKE, None) == B.MOE_ERR_UNSUPPORTED
    # null pointers, misaligned codes, a small workspace
    assert ffn(FAKE, None, *[FAKE] * 7, d, FAKE, FAKE, need, None) == B.MOE_ERR_INVALID
    assert ffn(*args9, d, None, FAKE, need, None) == B.MOE_ERR_INVALID
    assert ffn(FAKE, FAKE_MIS, *[FAKE] * 7, d, FAKE, FAKE, need, None) == B.MOE_ERR_UNSUPPORTED
    odd = ctypes.c_void_p(0x10001)
    assert ffn(FAKE, FAKE, odd, *[FAKE] * 6, d, FAKE, FAKE, need, None) == B.MOE_ERR_UNSUPPORTED
    assert ffn(*args9, d, FAKE, FAKE, need - 1, None) == B.MOE_ERR_WORKSPACE
    assert up(*[FAKE] * 7, d, FAKE, need - 1, None) == B.MOE_ERR_WORKSPACE
    assert down(FAKE, None, *[FAKE] * 5, d, need, FAKE, None) == B.MOE_ERR_INVALID
    # an empty batch launches nothing and touches no pointer
    d0 = B.dims(0, 2880, 128, 4, 2880)
    assert ffn(*[None] * 9, d0, None, None, 0, None) == B.MOE_OK


def test_mxfp4_pack_arguments_rejected(lib):
    pu, pd = lib.moe_pack_mxfp4_up, lib.moe_pack_mxfp4_down
    F2 = ctypes.c_void_p(0x20000)
    F3 = ctypes.c_void_p(0x30000)
    assert pu(FAKE, FAKE, FAKE, FAKE, -1, 16, 64, F2, F3, None) == B.MOE_ERR_INVALID
    assert pu(FAKE, FAKE, FAKE, FAKE, 2, 24, 64, F2, F3, None) == B.MOE_ERR_UNSUPPORTED   # I % 16
    assert pu(FAKE, FAKE, FAKE, FAKE, 2, 16, 96, F2, F3, None) == B.MOE_ERR_UNSUPPORTED   # H % 64
    assert pd(FAKE, FAKE, 2, 48, 64, F2, F3, None) == B.MOE_ERR_UNSUPPORTED               # H % 32
    assert pd(FAKE, FAKE, 2, 32, 96, F2, F3, None) == B.MOE_ERR_UNSUPPORTED               # I % 64
    assert pu(FAKE, None, FAKE, FAKE, 2, 16, 64, F2, F3, None) == B.MOE_ERR_INVALID
    assert pd(FAKE, FAKE, 2, 32, 64, FAKE, F3, None) == B.MOE_ERR_INVALID                 # in place
    assert pd(FAKE, FAKE, 2, 32, 64, FAKE_MIS, F3, None) == B.MOE_ERR_UNSUPPORTED         # codes out
    assert pu(FAKE, FAKE, FAKE, FAKE, 0, 16, 64, None, None, None) == B.MOE_OK            # nothing to do


def test_routed_up_validates_on_host(lib):
    # moe_expert_ffn_up_routed / _mxfp4: the dims, null, alignment and
    # workspace checks of moe_bucket and the up projection, before any launch.
    fns = (lambda d, ids=FAKE, cnt=FAKE, ws_bytes=1 << 40, x=FAKE:
           lib.moe_expert_ffn_up_routed(x, FAKE, ids, d, cnt, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                        ws_bytes, None),
           lambda d, ids=FAKE, cnt=FAKE, ws_bytes=1 << 40, x=FAKE:
           lib.moe_expert_ffn_mxfp4_up_routed(x, FAKE, FAKE, ids, d, cnt, FAKE, FAKE, FAKE, FAKE,
                                              FAKE, FAKE, ws_bytes, None))
    for f in fns:
        assert f(B.dims(64, 2048, 128, 129, 768)) == B.MOE_ERR_INVALID         # K > E
        assert f(B.dims(64, 2048, 257, 8, 768)) == B.MOE_ERR_UNSUPPORTED       # E above the limit
        assert f(B.dims(*GOOD), ids=None) == B.MOE_ERR_INVALID
        assert f(B.dims(*GOOD), cnt=None) == B.MOE_ERR_INVALID
        assert f(B.dims(*GOOD), x=None) == B.MOE_ERR_INVALID
        assert f(B.dims(*GOOD), ids=ctypes.c_void_p(0x10002)) == B.MOE_ERR_UNSUPPORTED
        assert f(B.dims(*GOOD), x=FAKE_MIS) == B.MOE_ERR_UNSUPPORTED
        d = B.dims(*GOOD)
        assert f(d, ws_bytes=B.moe_ffn_workspace_bytes(d) - 1) == B.MOE_ERR_WORKSPACE
    # MXFP4 reductions must be multiples of 64
    assert fns[1](B.dims(64, 2048 + 32, 128, 8, 768)) == B.MOE_ERR_UNSUPPORTED


def test_fused_ffn_validates_on_host(lib):
    # moe_expert_ffn_routed / _mxfp4: the sync buffer's null and alignment
    # checks, then those of moe_bucket and moe_expert_ffn, before any launch.
    def bf16(d, ids=FAKE, cnt=FAKE, ws_bytes=1 << 40, x=FAKE, y=FAKE, sync=FAKE, ws=FAKE):
        return lib.moe_expert_ffn_routed(x, FAKE, FAKE, ids, d, cnt, FAKE, FAKE, FAKE, FAKE, FAKE,
                                         y, ws, ws_bytes, sync, None)

    def mx(d, ids=FAKE, cnt=FAKE, ws_bytes=1 << 40, x=FAKE, y=FAKE, sync=FAKE, ws=FAKE):
        return lib.moe_expert_ffn_mxfp4_routed(x, FAKE, FAKE, FAKE, FAKE, ids, d, cnt, FAKE, FAKE,
                                               FAKE, FAKE, FAKE, y, ws, ws_bytes, sync, None)

    for f in (bf16, mx):
        assert f(B.dims(64, 2048, 128, 129, 768)) == B.MOE_ERR_INVALID         # K > E
        assert f(B.dims(64, 2048, 257, 8, 768)) == B.MOE_ERR_UNSUPPORTED       # E above the limit
        assert f(B.dims(*GOOD), sync=None) == B.MOE_ERR_INVALID
        assert f(B.dims(*GOOD), sync=ctypes.c_void_p(0x10002)) == B.MOE_ERR_UNSUPPORTED
        assert f(B.dims(*GOOD), ids=None) == B.MOE_ERR_INVALID
        assert f(B.dims(*GOOD), cnt=None) == B.MOE_ERR_INVALID
        assert f(B.dims(*GOOD), x=None) == B.MOE_ERR_INVALID
        assert f(B.dims(*GOOD), y=None) == B.MOE_ERR_INVALID
        assert f(B.dims(*GOOD), ids=ctypes.c_void_p(0x10002)) == B.MOE_ERR_UNSUPPORTED
        assert f(B.dims(*GOOD), y=FAKE_MIS) == B.MOE_ERR_UNSUPPORTED
        # h rows must be whole 128-byte lines for the in-launch hand-over
        assert f(B.dims(*GOOD), ws=ctypes.c_void_p(0x10010)) == B.MOE_ERR_UNSUPPORTED
        d = B.dims(*GOOD)
        assert f(d, ws_bytes=B.moe_ffn_workspace_bytes(d) - 1) == B.MOE_ERR_WORKSPACE
    assert mx(B.dims(64, 2048 + 32, 128, 8, 768)) == B.MOE_ERR_UNSUPPORTED
    assert lib.moe_ffn_sync_bytes(B.dims(*GOOD)) == 4 * (64 * 128 + 1)
    assert lib.moe_ffn_sync_bytes(B.dims(64, 2048, 128, 129, 768)) == 0


def test_noalloc_ffn_rejects_oversize_on_host(lib):
    # The fixed workspace holds 32 MiB; a larger problem is refused before the
    # library touches a device.
    assert lib.moe_expert_ffn_noalloc_max_bytes() == 32 << 20
    d = B.dims(4096, 2048, 128, 16, 768)  # T*K*I*4 = 201 MB
    assert lib.moe_expert_ffn_noalloc(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, d, FAKE,
                                      None) == B.MOE_ERR_WORKSPACE
    assert lib.moe_expert_ffn_noalloc(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                      B.dims(64, 2048, 128, 129, 768), FAKE, None) == B.MOE_ERR_INVALID
    assert lib.moe_expert_ffn_noalloc(None, None, None, None, None, None, None,
                                      B.dims(0, 2048, 128, 8, 768), None, None) == B.MOE_OK
