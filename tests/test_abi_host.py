"""C-ABI checks that need no GPU: exported symbols, validation error codes,
and the packed prefix layout against a numpy gather (CPU only)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2609_10018_amd import ffi, inputs
from paper_2609_10018_amd.inputs import CONFIGS, DNTable

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "elasto.h")


@pytest.fixture(scope="module")
def lib():
    return ffi.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(elasto_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function(lib):
    names = declared_functions()
    assert "elasto_create" in names and "elasto_forward" in names and "elasto_set_mode" in names
    for n in names:
        assert hasattr(lib, n), n


def _table_copy(t):
    return DNTable(t.n_heads.copy(), t.n_mlp.copy(), t.head_order.copy(), t.mlp_order.copy(),
                   t.n_embed.copy(), t.embed_order.copy())


@pytest.mark.parametrize("name", list(CONFIGS))
def test_valid_tables_pass(lib, name):
    cfg = CONFIGS[name]
    assert ffi.validate(cfg, inputs.make_dn_table(cfg), cfg.batch) == 0


def test_bad_tables_rejected(lib):
    cfg = CONFIGS["vit_ti"]
    base = inputs.make_dn_table(cfg)
    bad = []
    t = _table_copy(base); t.n_heads[1, 3] = 0; bad.append(t)
    t = _table_copy(base); t.n_heads[0, 0] = cfg.heads + 1; bad.append(t)
    t = _table_copy(base); t.n_mlp[2, 5] = cfg.mlp_hidden + 1; bad.append(t)
    t = _table_copy(base); t.n_mlp[2, 5] = -3; bad.append(t)
    t = _table_copy(base); t.head_order[4, 0] = t.head_order[4, 1]; bad.append(t)
    t = _table_copy(base); t.mlp_order[0, 7] = cfg.mlp_hidden; bad.append(t)
    t = DNTable(base.n_heads[:, :5].copy(), base.n_mlp[:, :5].copy(), base.head_order[:5].copy(),
                base.mlp_order[:5].copy()); bad.append(t)
    t = _table_copy(base); t.n_embed[1] = 0; bad.append(t)
    t = _table_copy(base); t.n_embed[1] = cfg.dim + 8; bad.append(t)
    t = _table_copy(base); t.n_embed[2] = 100; bad.append(t)          # bf16: not a multiple of 8
    t = _table_copy(base); t.embed_order[3] = t.embed_order[4]; bad.append(t)
    for t in bad:
        assert ffi.validate(cfg, t, 4) == 3, ffi.last_error()
        assert ffi.last_error()


@pytest.mark.parametrize("change,code", [
    (dict(dim=190), 2),                # dim % heads != 0
    (dict(img=220), 2),                # img % patch != 0
    (dict(heads=4), 2),                # bf16 head_dim 48 != 64
    (dict(patch=12, img=216), 2),      # bf16 patch % 8 != 0
    (dict(mlp_hidden=0), 2),
    (dict(ln_eps=0.0), 2),
    (dict(dtype=7), 2),
])
def test_bad_configs_rejected(lib, change, code):
    import dataclasses
    cfg = dataclasses.replace(CONFIGS["vit_ti"], **change)
    table = inputs.make_dn_table(CONFIGS["vit_ti"])
    assert ffi.validate(cfg, table, 4) == code


def test_create_rejects_before_any_hip_call(lib):
    cfg = CONFIGS["tiny"]
    w = inputs.make_weights(cfg)
    t = inputs.make_dn_table(cfg)
    t.n_heads[1, 0] = 5
    with pytest.raises(ffi.ElastoError) as e:
        ffi.ElasticViT(cfg, w, t, 4)
    assert e.value.status == 3
    import dataclasses
    with pytest.raises(ffi.ElastoError) as e:
        ffi.ElasticViT(dataclasses.replace(cfg, dim=63), w, inputs.make_dn_table(cfg), 4)
    assert e.value.status == 2


def test_null_handle_calls_fail_cleanly(lib):
    assert lib.elasto_set_mode(None, 0) == 1
    assert lib.elasto_forward(None, None, 1, None, None) == 1
    assert lib.elasto_destroy(None) == 0
    k = ctypes.c_int32()
    assert lib.elasto_get_mode(None, ctypes.byref(k)) == 1


def _view(buf, cfg, tensor, layer=0):
    off, rows, cols, eb = ffi.packed_layout(cfg, tensor, layer)
    assert off % 256 == 0
    if eb == 2:
        raw = buf[off:off + rows * cols * 2].view(np.uint16).reshape(rows, cols)
        return (raw.astype(np.uint32) << 16).view(np.float32)
    return buf[off:off + rows * cols * 4].view(np.float32).reshape(rows, cols)


@pytest.mark.parametrize("name", ["tiny", "vit_ti", "vit_ti_emb"])
def test_pack_equals_numpy_gather(lib, name):
    cfg = CONFIGS[name]
    w = inputs.make_weights(cfg)
    t = inputs.make_dn_table(cfg)
    buf = ffi.pack_weights(cfg, w, t)
    sw = inputs.stored_weights(cfg, w)      # bf16-rounded matrices on the bf16 path
    d, hd, H = cfg.dim, cfg.head_dim, cfg.heads
    ev = t.embed_order                      # packed embedding channel j = canonical ev[j]
    np.testing.assert_array_equal(_view(buf, cfg, ffi.T_PATCH_W), sw["patch_w"].reshape(d, -1)[ev])
    np.testing.assert_array_equal(_view(buf, cfg, ffi.T_POS), sw["pos"][:, ev])
    np.testing.assert_array_equal(_view(buf, cfg, ffi.T_HEAD_W), sw["head_w"][:, ev])
    np.testing.assert_array_equal(_view(buf, cfg, ffi.T_CLS)[0], sw["cls"][ev])
    np.testing.assert_array_equal(_view(buf, cfg, ffi.T_NORM_G)[0], sw["norm_g"][ev])
    for l in range(cfg.depth):
        ho, mo = t.head_order[l], t.mlp_order[l]
        rows = np.array([tq * d + ho[s] * hd + c for s in range(H) for tq in range(3)
                         for c in range(hd)])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_WQKV, l), sw["qkv_w"][l][rows][:, ev])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_BQKV, l)[0], sw["qkv_b"][l][rows])
        cols = np.array([ho[s] * hd + c for s in range(H) for c in range(hd)])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_WO, l), sw["proj_w"][l][ev][:, cols])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_BO, l)[0], sw["proj_b"][l][ev])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_W1, l), sw["fc1_w"][l][mo][:, ev])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_B1, l)[0], sw["fc1_b"][l][mo])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_W2, l), sw["fc2_w"][l][ev][:, mo])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_B2, l)[0], sw["fc2_b"][l][ev])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_LN1_B, l)[0], sw["ln1_b"][l][ev])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_LN2_G, l)[0], sw["ln2_g"][l][ev])


@pytest.mark.parametrize("name", ["vit_ti", "vit_ti_emb"])
def test_packed_prefix_is_what_mode_k_reads(lib, name):
    """The first n rows of WQKV / W1 are exactly mode k's active heads / units,
    and the first n_embed[k] embedding positions its active channels."""
    cfg = CONFIGS[name]
    w = inputs.make_weights(cfg)
    t = inputs.make_dn_table(cfg)
    buf = ffi.pack_weights(cfg, w, t)
    sw = inputs.stored_weights(cfg, w)
    import oracle
    for k in range(t.num_modes):
        p = oracle.extract_dense(sw, cfg, t, k)
        E = int(t.n_embed[k])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_PATCH_W)[:E],
                                      p["patch_w"].reshape(E, -1))
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_POS)[:, :E], p["pos"])
        np.testing.assert_array_equal(_view(buf, cfg, ffi.T_HEAD_W)[:, :E], p["head_w"])
        for l in range(cfg.depth):
            h, m = int(t.n_heads[k, l]), int(t.n_mlp[k, l])
            lp = p["layers"][l]
            np.testing.assert_array_equal(_view(buf, cfg, ffi.T_W1, l)[:m, :E], lp["fc1_w"])
            np.testing.assert_array_equal(_view(buf, cfg, ffi.T_W2, l)[:E, :m], lp["fc2_w"])
            wo = _view(buf, cfg, ffi.T_WO, l)[:E, :h * cfg.head_dim]
            np.testing.assert_array_equal(wo, lp["proj_w"])
            packed_q = _view(buf, cfg, ffi.T_WQKV, l)[:3 * cfg.head_dim * h, :E]
            pq = packed_q.reshape(h, 3, cfg.head_dim, E).transpose(1, 0, 2, 3)
            np.testing.assert_array_equal(pq.reshape(-1, E), lp["qkv_w"])
            np.testing.assert_array_equal(_view(buf, cfg, ffi.T_LN1_G, l)[0, :E], lp["ln1_g"])


def test_bf16_rounding_agrees_with_numpy_rne(lib):
    cfg = CONFIGS["vit_ti"]
    w = inputs.make_weights(cfg)
    rng = np.random.default_rng(3)
    special = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -0.0, 65504.0, 1e-40, 3.3895e38],
                       dtype=np.float32)
    w["head_w"] = w["head_w"].copy()
    w["head_w"].reshape(-1)[:special.size] = special
    w["head_w"].reshape(-1)[special.size:special.size + 100] = rng.standard_normal(100) * 1e3
    t = inputs.make_dn_table(cfg)
    buf = ffi.pack_weights(cfg, w, t)
    np.testing.assert_array_equal(_view(buf, cfg, ffi.T_HEAD_W),
                                  inputs.bf16_round(w["head_w"])[:, t.embed_order])


def test_op_entry_points_validate_before_any_hip_call(lib):
    """Shape and alignment checks of the single-kernel entry points return
    INVALID_ARG without touching the (fake, never dereferenced) pointers."""
    p16 = ctypes.c_void_p(1 << 20)
    p8 = ctypes.c_void_p((1 << 20) + 8)
    f = ctypes.c_float(1e-6)
    ln = lib.elasto_op_layernorm
    # bf16 LayerNorm: d and the stride must be multiples of 8, pointers 16-byte aligned
    assert ln(1, p16, 12, None, 1, p16, 4, 12, p16, p16, f, None) == 1
    assert ln(1, p16, 772, None, 1, p16, 4, 768, p16, p16, f, None) == 1
    assert ln(1, p8, 768, None, 1, p16, 4, 768, p16, p16, f, None) == 1
    assert ln(1, p16, 768, None, 1, p8, 4, 768, p16, p16, f, None) == 1
    assert ln(1, p16, 768, None, 1, p16, 4, 4096, p16, p16, f, None) == 1   # d > 2048
    assert ln(0, p16, 768, p16, 197, p16, 4, 768, p16, p16, f, None) == 1   # x_cls needs bf16
    assert ln(1, p16, 768, p16, 0, p16, 4, 768, p16, p16, f, None) == 1     # tokens >= 1
    assert lib.elasto_last_error()
    # bf16 attention: head_dim 64, tokens <= 240, qkv 16-byte and o 8-byte aligned,
    # o_stride a multiple of 4 covering every head slot, the o range of one
    # sequence below 2^31 bytes
    at = lib.elasto_op_attention
    p4 = ctypes.c_void_p((1 << 20) + 4)
    s = ctypes.c_float(0.125)
    assert at(1, p16, 384, p16, 128, 2, 197, 2, 32, s, None) == 1          # head_dim
    assert at(1, p16, 384, p16, 128, 2, 241, 2, 64, s, None) == 1          # tokens
    assert at(1, p8, 384, p16, 128, 2, 197, 2, 64, s, None) == 1           # qkv alignment
    assert at(1, p16, 384, p4, 128, 2, 197, 2, 64, s, None) == 1           # o alignment
    assert at(1, p16, 384, p16, 130, 2, 197, 2, 64, s, None) == 1          # o_stride % 4
    assert at(1, p16, 384, p16, 64, 2, 197, 2, 64, s, None) == 1           # o_stride < heads * 64
    assert at(1, p16, 384, p16, 1 << 23, 2, 240, 2, 64, s, None) == 1      # o range >= 2^31
    assert at(1, p16, 320, p16, 128, 2, 197, 2, 64, s, None) == 1          # qkv_stride < 3 heads 64


def test_conv2d_validates_before_any_hip_call(lib):
    """Channel counts, strides, alignment and the 2 GiB range-check limit are
    refused with INVALID_ARG before any pointer is used."""
    p16 = ctypes.c_void_p(1 << 20)
    p8 = ctypes.c_void_p((1 << 20) + 8)
    cv = lib.elasto_op_conv2d

    def call(x=p16, batch=2, H=14, W=14, cs=64, ca=64, kh=3, kw=3, stride=1, pad=1, w=p16,
             ldw=576, wseg=64, bias=p16, y=p16, ldy=64, n=64, relu=1):
        return cv(x, batch, H, W, cs, ca, kh, kw, stride, pad, w, ldw, wseg, bias, y, ldy, n,
                  relu, None)

    assert call(ca=60) == 1                 # channel prefix not a multiple of 8
    assert call(ca=0) == 1
    assert call(ca=72) == 1                 # more active channels than stored
    assert call(wseg=56) == 1               # tap segment shorter than the prefix
    assert call(ldw=568) == 1               # rows shorter than kh*kw*wseg
    assert call(ldy=60) == 1
    assert call(n=0) == 1
    assert call(stride=0) == 1
    assert call(H=1, pad=0) == 1            # kernel larger than the padded image
    assert call(x=p8) == 1
    assert call(y=p8) == 1
    assert call(x=None) == 1
    assert call(H=4096, W=4096, cs=128, ca=128, ldw=1152, wseg=128) == 1  # one image > 2 GiB
    assert lib.elasto_last_error()



def test_cnn_validation_rejects_bad_shapes_and_tables():
    """elasto_cnn_validate: the shipped configs pass; bad image sizes, channel
    counts and widths give BAD_CONFIG, bad DN tables BAD_TABLE."""
    import dataclasses
    from paper_2609_10018_amd.inputs_cnn import CNN_CONFIGS, make_cnn_table
    for name in CNN_CONFIGS:
        assert ffi.cnn_validate(CNN_CONFIGS[name], make_cnn_table(CNN_CONFIGS[name])) == 0
    cfg = CNN_CONFIGS["resnet_small"]
    t = make_cnn_table(cfg)
    for change in ({"img": 48}, {"in_chans": 5}, {"in_chans": 0}, {"stem": 12},
                   {"widths": (16, 32, 60, 128)}):
        assert ffi.cnn_validate(dataclasses.replace(cfg, **change), t) == 2, change
    bad = make_cnn_table(cfg)
    bad.n_width[1, 0] = 12                      # not a multiple of 8
    assert ffi.cnn_validate(cfg, bad) == 3
    bad = make_cnn_table(cfg)
    bad.n_width[0, 2] = cfg.block_specs()[2]["width"] + 8   # wider than the block
    assert ffi.cnn_validate(cfg, bad) == 3
    bad = make_cnn_table(cfg)
    bad.order2[1][0] = bad.order2[1][1]         # not a permutation
    assert ffi.cnn_validate(cfg, bad) == 3
