"""The C ABI on the CPU: the library loads, exports every symbol the header
declares, and rejects invalid arguments before anything is launched.

Only argument combinations that fail validation are passed here, so no HIP
kernel or device call is ever reached (the fake pointers below are never
dereferenced).
"""

import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cardan.h")


@pytest.fixture(scope="module")
def C():
    from paper_2609_21137_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    from paper_2609_21137_amd import cardan
    return cardan


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(cardan_[a-z0-9_]+)\s*\(", text)))


def test_header_symbols_exported(C):
    names = _declared()
    assert len(names) >= 10
    out = subprocess.run(["nm", "-D", "--defined-only", C.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (cardan_\w+)", out))
    for n in names:
        assert n in exported, n
        assert hasattr(C.lib(), n)
    assert set(C.EXPORTED) == set(names)


def test_abi_version(C):
    assert C.abi_version() == 1
    m = re.search(r"#define CARDAN_ABI_VERSION (\d+)", open(HEADER).read())
    assert int(m.group(1)) == C.abi_version()


def _ws(C, shape, B):
    n = ctypes.c_size_t(0)
    rc = C.lib().cardan_workspace_bytes(ctypes.byref(shape), B, ctypes.byref(n))
    return rc, n.value


def test_workspace_bytes(C):
    from paper_2609_21137_amd.configs import QWEN3_B1, QWEN3_B16, TINY, WIDE_SKEW_B4
    for w in (TINY, QWEN3_B1, QWEN3_B16, WIDE_SKEW_B4):
        rc, n = _ws(C, C.shape_of(w), w.B)
        assert rc == 0 and n > 0 and n % 256 == 0
    s = C.shape_of(QWEN3_B1)
    sizes = [_ws(C, s, B)[1] for B in (1, 2, 4, 8, 16, 32, 64)]
    assert sizes == sorted(sizes)
    assert C.workspace_bytes(s, 16) == sizes[4]


BAD_SHAPES = [
    # (H, I, E, top_k, d, K, r, B, expected code)
    ((2048, 768, 128, 8, 8, 256, 128), 0, -2),
    ((2048, 768, 128, 8, 8, 256, 128), 65, -2),
    ((2048, 768, 8, 9, 8, 256, 128), 1, -2),      # top_k > E
    ((2048, 770, 128, 8, 8, 256, 128), 1, -2),    # I % d
    ((2048, 768, 128, 8, 8, 300, 128), 1, -2),    # K > 256
    ((2048, 768, 128, 8, 16, 256, 128), 1, -3),   # d = 16 not compiled
    ((2016, 768, 128, 8, 8, 256, 128), 1, -3),    # H % 64
    ((2048, 784, 128, 8, 8, 256, 128), 1, -3),    # I % 32
    ((2048, 768, 128, 8, 8, 256, 12), 1, -3),     # r % 8
    ((2048, 768, 2048, 8, 8, 256, 128), 1, -3),   # E > 1024
    ((2048, 768, 128, 40, 8, 256, 128), 1, -3),   # top_k > 32
    ((0, 768, 128, 8, 8, 256, 128), 1, -2),
]


@pytest.mark.parametrize("dims,B,code", BAD_SHAPES)
def test_bad_shapes(C, dims, B, code):
    rc, _ = _ws(C, C.make_shape(*dims), B)
    assert rc == code, C.lib().cardan_last_error()
    assert C.lib().cardan_last_error()


def test_null_shape_and_out(C):
    L = C.lib()
    assert L.cardan_workspace_bytes(None, 1, ctypes.byref(ctypes.c_size_t())) == -1
    s = C.make_shape(2048, 768, 128, 8, 8, 256, 128)
    assert L.cardan_workspace_bytes(ctypes.byref(s), 1, None) == -1


FAKE = 0x10000          # aligned, never dereferenced: every call below fails validation


def _layer(C, **over):
    vals = {n: FAKE for n in C.LAYER_FIELDS}
    vals.update(over)
    return C.LayerStruct(*[vals[n] for n in C.LAYER_FIELDS])


def test_moe_layer_validation(C):
    L = C.lib()
    s = C.make_shape(2048, 768, 128, 8, 8, 256, 128)
    lay = _layer(C)
    _, need = _ws(C, s, 1)
    # NULL x
    assert L.cardan_moe_layer(ctypes.byref(s), 1, None, ctypes.byref(lay), FAKE, FAKE, FAKE,
                              FAKE, need, None) == -1
    # misaligned x
    assert L.cardan_moe_layer(ctypes.byref(s), 1, FAKE + 2, ctypes.byref(lay), FAKE, FAKE, FAKE,
                              FAKE, need, None) == -6
    # NULL layer
    assert L.cardan_moe_layer(ctypes.byref(s), 1, FAKE, None, FAKE, FAKE, FAKE, FAKE, need,
                              None) == -1
    # NULL code book
    bad = _layer(C, cb_down=None)
    assert L.cardan_moe_layer(ctypes.byref(s), 1, FAKE, ctypes.byref(bad), FAKE, FAKE, FAKE,
                              FAKE, need, None) == -1
    assert b"cb_down" in L.cardan_last_error()
    # NULL low-rank factor with r > 0
    bad = _layer(C, A_down=None)
    assert L.cardan_moe_layer(ctypes.byref(s), 1, FAKE, ctypes.byref(bad), FAKE, FAKE, FAKE,
                              FAKE, need, None) == -1
    # workspace too small, NULL, misaligned
    assert L.cardan_moe_layer(ctypes.byref(s), 1, FAKE, ctypes.byref(lay), FAKE, FAKE, FAKE,
                              FAKE, 256, None) == -4
    assert L.cardan_moe_layer(ctypes.byref(s), 1, FAKE, ctypes.byref(lay), FAKE, FAKE, FAKE,
                              None, need, None) == -1
    assert L.cardan_moe_layer(ctypes.byref(s), 1, FAKE, ctypes.byref(lay), FAKE, FAKE, FAKE,
                              FAKE + 8, need, None) == -6
    # bad batch
    assert L.cardan_moe_layer(ctypes.byref(s), 0, FAKE, ctypes.byref(lay), FAKE, FAKE, FAKE,
                              FAKE, need, None) == -2


def test_other_entry_points_validation(C):
    L = C.lib()
    s = C.make_shape(2048, 768, 128, 8, 8, 256, 128)
    _, need = _ws(C, s, 4)
    assert L.cardan_route_topk(ctypes.byref(s), 4, FAKE, None, None, FAKE, FAKE, FAKE, need,
                               None) == -1
    assert L.cardan_route_topk(ctypes.byref(s), 4, FAKE, FAKE, FAKE + 2, FAKE, FAKE, FAKE, need,
                               None) == -6
    assert L.cardan_route_topk(ctypes.byref(s), 4, FAKE, FAKE, None, FAKE, FAKE, FAKE, 16,
                               None) == -4
    s0 = C.make_shape(2048, 768, 128, 8, 8, 256, 0)
    assert L.cardan_shared_proj(ctypes.byref(s0), 4, FAKE, FAKE, FAKE, FAKE, FAKE, need,
                                None) == -2
    assert L.cardan_shared_proj(ctypes.byref(s), 4, FAKE, FAKE, FAKE, None, FAKE, need,
                                None) == -1
    lay = _layer(C)
    assert L.cardan_vq_lr_expert_ffn(ctypes.byref(s), 4, FAKE, FAKE, FAKE, None,
                                     ctypes.byref(lay), FAKE, FAKE, need, None) == -1
    assert L.cardan_vq_lr_expert_ffn(ctypes.byref(s), 4, FAKE, FAKE, FAKE, FAKE,
                                     ctypes.byref(lay), FAKE, FAKE, 0, None) == -4
    assert L.cardan_rmsnorm_bf16(0, 2048, FAKE, 1e-6, FAKE, None) == -2
    assert L.cardan_rmsnorm_bf16(4, 2048, None, 1e-6, FAKE, None) == -1
    assert L.cardan_profile_begin(0) == -2
    assert L.cardan_profile_end(None, None) == -1


def test_binding_rejects_host_tensors(C):
    import torch
    s = C.make_shape(256, 128, 8, 2, 4, 16, 8)
    x = torch.zeros((1, 256), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        C._ptr(x, torch.bfloat16, "x")
    with pytest.raises(ValueError):
        C._ptr(torch.zeros(3, dtype=torch.float32), torch.bfloat16, "x")
    del s


def _dense(C, **over):
    vals = {n: FAKE for n in C.DENSE_LAYER_FIELDS}
    vals.update(over)
    return C.DenseLayerStruct(*[vals[n] for n in C.DENSE_LAYER_FIELDS])


def test_dense_entry_points_validation(C):
    L = C.lib()
    s = C.make_shape(2048, 768, 128, 8, 8, 256, 128)
    _, need = _ws(C, s, 1)
    lay = _layer(C)
    # dense down: the compressed down fields may be NULL, W_down may not
    nodown = _layer(C, cb_down=None, codes_down=None, A_down=None, B_down=None)
    assert L.cardan_moe_layer_dense_down(ctypes.byref(s), 1, FAKE, ctypes.byref(nodown), None,
                                         FAKE, FAKE, FAKE, FAKE, need, None) == -1
    assert b"W_down" in L.cardan_last_error()
    assert L.cardan_moe_layer_dense_down(ctypes.byref(s), 1, FAKE, ctypes.byref(nodown), FAKE + 4,
                                         FAKE, FAKE, FAKE, FAKE, need, None) == -6
    assert L.cardan_moe_layer_dense_down(ctypes.byref(s), 1, FAKE, ctypes.byref(nodown), FAKE,
                                         FAKE, FAKE, FAKE, FAKE, 256, None) == -4
    bad = _layer(C, V_up=None)  # gate/up factors are still required
    assert L.cardan_moe_layer_dense_down(ctypes.byref(s), 1, FAKE, ctypes.byref(bad), FAKE,
                                         FAKE, FAKE, FAKE, FAKE, need, None) == -1
    assert L.cardan_moe_layer_dense_down(ctypes.byref(s), 65, FAKE, ctypes.byref(lay), FAKE,
                                         FAKE, FAKE, FAKE, FAKE, need, None) == -2
    # uncompressed layer: d, K and r of the shape are not read
    dl = _dense(C)
    s_any = C.make_shape(2048, 768, 128, 8, 0, 0, 0)
    for field in ("router_w", "W_gate", "W_up", "W_down"):
        assert L.cardan_dense_moe_layer(ctypes.byref(s_any), 1, FAKE, ctypes.byref(_dense(C, **{field: None})),
                                        FAKE, FAKE, FAKE, FAKE, need, None) == -1
        assert field.encode() in L.cardan_last_error()
    assert L.cardan_dense_moe_layer(ctypes.byref(s_any), 1, FAKE, ctypes.byref(_dense(C, router_bias=FAKE + 2)),
                                    FAKE, FAKE, FAKE, FAKE, need, None) == -6
    assert L.cardan_dense_moe_layer(ctypes.byref(s_any), 1, FAKE, None, FAKE, FAKE, FAKE, FAKE, need,
                                    None) == -1
    assert L.cardan_dense_moe_layer(None, 1, FAKE, ctypes.byref(dl), FAKE, FAKE, FAKE, FAKE, need,
                                    None) == -1
    assert L.cardan_dense_moe_layer(ctypes.byref(s_any), 1, FAKE, ctypes.byref(dl), FAKE, FAKE, FAKE,
                                    FAKE, 256, None) == -4
    big = C.make_shape(65536, 16384, 128, 8, 8, 256, 0)  # one expert matrix of 2 GiB
    assert L.cardan_dense_moe_layer(ctypes.byref(big), 1, FAKE, ctypes.byref(dl), FAKE, FAKE, FAKE,
                                    FAKE, need, None) == -3


def test_workspace_covers_dense_forms(C):
    """The workspace size is the maximum over the compressed, dense-down and
    uncompressed layouts, whatever d, K and r the size query names."""
    for dims in ((2048, 768, 128, 8, 8, 256, 128), (2048, 768, 128, 8, 4, 16, 0)):
        s = C.make_shape(*dims)
        for B in (1, 16):
            assert _ws(C, s, B)[0] == 0
    a = _ws(C, C.make_shape(2048, 768, 128, 8, 8, 256, 128), 16)[1]
    b = _ws(C, C.make_shape(2048, 768, 128, 8, 8, 256, 0), 16)[1]
    assert a >= b > 0


def test_noalloc_validation(C):
    """The no-allocation entry point validates before touching a device: a
    NULL argument, a bad shape and a layer whose workspace exceeds the
    library's scratch array are refused."""
    lib = C.lib()
    fake = ctypes.c_void_p(0x100000)  # 16-byte aligned, never dereferenced
    st = C.LayerStruct(*([0x100000] * len(C.LAYER_FIELDS)))
    qwen = C.make_shape(2048, 768, 128, 8, 8, 256, 128)
    assert lib.cardan_moe_layer_noalloc(None, 1, fake, ctypes.byref(st), fake, fake, fake, None) == -1
    assert lib.cardan_moe_layer_noalloc(ctypes.byref(qwen), 1, None, ctypes.byref(st), fake, fake, fake,
                                        None) == -1
    assert lib.cardan_moe_layer_noalloc(ctypes.byref(qwen), 0, fake, ctypes.byref(st), fake, fake, fake,
                                        None) == -2
    wide = C.make_shape(4096, 1536, 64, 6, 8, 256, 256)
    rc = lib.cardan_moe_layer_noalloc(ctypes.byref(wide), 64, fake, ctypes.byref(st), fake, fake, fake, None)
    assert rc == -4, lib.cardan_last_error().decode()
    assert b"scratch" in lib.cardan_last_error()
