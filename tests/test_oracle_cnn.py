"""Pins of the elastic-ResNet oracle against things other than itself (CPU):
brute-force convolution / pooling loops, a textbook network from torch fp64
library ops (full width, and every mode on weights masked kernel by kernel),
mask form vs gather form, locality, and the MAC counts of Table 2."""
import numpy as np
import pytest

from oracle import resnet as orn
from paper_2609_10018_amd import cost
from paper_2609_10018_amd.inputs_cnn import (CNN_CONFIGS, make_cnn_images, make_cnn_table,
                                             make_cnn_weights)
from textbook import rel_err
from textbook_cnn import loop_masked_cnn_weights, torch_resnet

SMALL = CNN_CONFIGS["resnet_small"]


@pytest.mark.parametrize("k,stride,pad", [(1, 1, 0), (3, 1, 1), (3, 2, 1), (7, 2, 3), (1, 2, 0)])
def test_conv2d_matches_loop(k, stride, pad):
    rng = np.random.default_rng(k * 10 + stride)
    x = rng.standard_normal((2, 3, 9, 9))
    w = rng.standard_normal((4, 3, k, k))
    b = rng.standard_normal(4)
    got = orn.conv2d(x, w, b, stride, pad)
    Ho = (9 + 2 * pad - k) // stride + 1
    ref = np.zeros((2, 4, Ho, Ho))
    for n in range(2):
        for o in range(4):
            for oh in range(Ho):
                for ow in range(Ho):
                    acc = b[o]
                    for c in range(3):
                        for i in range(k):
                            for j in range(k):
                                ih, iw = oh * stride - pad + i, ow * stride - pad + j
                                if 0 <= ih < 9 and 0 <= iw < 9:
                                    acc += x[n, c, ih, iw] * w[o, c, i, j]
                    ref[n, o, oh, ow] = acc
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_max_pool_matches_loop():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 3, 9, 8))
    got = orn.max_pool_3x3_s2(x)
    ref = np.zeros((2, 3, 5, 4))
    for oh in range(5):
        for ow in range(4):
            win = [x[:, :, ih, iw] for ih in range(2 * oh - 1, 2 * oh + 2)
                   for iw in range(2 * ow - 1, 2 * ow + 2) if 0 <= ih < 9 and 0 <= iw < 8]
            ref[:, :, oh, ow] = np.max(np.stack(win), axis=0)
    np.testing.assert_array_equal(got, ref)


def test_full_width_equals_textbook():
    w = make_cnn_weights(SMALL)
    x = make_cnn_images(SMALL, 3)
    got = orn.resnet_forward(orn.canonical_params(w, SMALL), x)
    assert rel_err(got, torch_resnet(w, x, SMALL)) < 1e-10
    # the logits depend on the image (white-noise images through a random
    # network give a large class-dependent common part; the image-dependent
    # part is still ~10% of the spread)
    assert np.abs(got - got.mean(axis=0)).max() > 0.02 * np.abs(got).max()


def test_every_mode_equals_textbook_on_loop_masked_weights():
    w = make_cnn_weights(SMALL)
    x = make_cnn_images(SMALL, 2)
    table = make_cnn_table(SMALL)
    for k in range(table.num_modes):
        ref = torch_resnet(loop_masked_cnn_weights(w, SMALL, table, k), x, SMALL)
        assert rel_err(orn.elastic_forward(w, SMALL, table, k, x), ref) < 1e-10, k
        assert rel_err(orn.elastic_forward_masked(w, SMALL, table, k, x), ref) < 1e-10, k


def test_resnet50_mask_form_equals_gather_form():
    cfg = CNN_CONFIGS["resnet50"]
    w = make_cnn_weights(cfg)
    x = make_cnn_images(cfg, 1)
    table = make_cnn_table(cfg)
    for k in (0, 3, 5):
        f2 = orn.elastic_forward_masked(w, cfg, table, k, x)
        f13 = orn.elastic_forward(w, cfg, table, k, x)
        assert rel_err(f13, f2) < 1e-10, k


def test_locality_of_pruned_filters():
    w = make_cnn_weights(SMALL)
    x = make_cnn_images(SMALL, 2)
    table = make_cnn_table(SMALL)
    k = 3
    w2 = {key: np.array(v, copy=True) for key, v in w.items()}
    for i, spec in enumerate(SMALL.block_specs()):
        a1, a2 = orn.active_filters(table, k, i)
        off1 = np.setdiff1d(np.arange(spec["width"]), a1)
        off2 = np.setdiff1d(np.arange(spec["width"]), a2)
        w2[f"b{i}_c1_w"][off1] = 5.0
        w2[f"b{i}_c1_b"][off1] = 5.0
        w2[f"b{i}_c2_w"][:, off1] = -3.0
        w2[f"b{i}_c2_w"][off2] = 2.0
        w2[f"b{i}_c2_b"][off2] = 2.0
        w2[f"b{i}_c3_w"][:, off2] = 7.0
    a = orn.elastic_forward(w, SMALL, table, k, x)
    assert np.array_equal(a, orn.elastic_forward(w2, SMALL, table, k, x))
    assert not np.array_equal(orn.elastic_forward(w, SMALL, table, 0, x),
                              orn.elastic_forward(w2, SMALL, table, 0, x))


def test_resnet50_macs_match_table2():
    """Full ResNet-50: 4.09 G MACs per image (the paper's Table 2 quotes 4.12 G);
    the six modes land within 2% of the paper's six DN levels."""
    cfg = CNN_CONFIGS["resnet50"]
    table = make_cnn_table(cfg)
    got = [cost.cnn_macs(cfg, table, k) / 1e9 for k in range(table.num_modes)]
    paper = [4.12, 3.33, 2.65, 2.03, 1.51, 1.07]
    assert got[0] == pytest.approx(4.089, abs=1e-3)
    for g, t in zip(got, paper):
        assert abs(g - t) / t < 0.02, (g, t)
    assert all(a > b for a, b in zip(got, got[1:]))


def test_cnn_macs_equal_direct_count_of_the_dense_network():
    w = make_cnn_weights(SMALL)
    table = make_cnn_table(SMALL)
    for k in range(table.num_modes):
        p = orn.extract_dense(w, SMALL, table, k)
        hw = SMALL.img // 2
        direct = hw * hw * p["stem"][0].size
        hw //= 2
        for blk, spec in zip(p["blocks"], SMALL.block_specs()):
            ho = hw // blk["stride"]
            direct += hw * hw * blk["c1"][0].size + ho * ho * blk["c2"][0].size
            direct += ho * ho * blk["c3"][0].size
            if "dn" in blk:
                direct += ho * ho * blk["dn"][0].size
            hw = ho
        direct += p["fc"][0].size
        assert cost.cnn_macs(SMALL, table, k) == direct


def _pool_no_pad(x):
    N, C, H, W = x.shape
    Ho, Wo = (H - 3) // 2 + 1, (W - 3) // 2 + 1
    out = np.full((N, C, Ho, Wo), -np.inf)
    for i in range(3):
        for j in range(3):
            out = np.maximum(out, x[:, :, i:i + 2 * Ho:2, j:j + 2 * Wo:2])
    return out


def _conv_flipped(x, w, b, stride, pad):
    return _orig_conv(x, w[:, :, ::-1, ::-1].copy(), b, stride, pad)


def _active_suffix(table, k, block):
    n = int(table.n_width[k][block])
    W = len(table.order1[block])
    return (np.asarray(table.order1[block][W - n:], dtype=np.int64),
            np.asarray(table.order2[block][W - n:], dtype=np.int64))


_orig_conv = orn.conv2d


@pytest.mark.parametrize("name,mutant", [("max_pool_3x3_s2", _pool_no_pad),
                                         ("conv2d", _conv_flipped),
                                         ("active_filters", _active_suffix)])
def test_cnn_pins_catch_planted_mistake(monkeypatch, name, mutant):
    w = make_cnn_weights(SMALL)
    x = make_cnn_images(SMALL, 2)
    table = make_cnn_table(SMALL)

    def worst():
        errs = [rel_err(orn.resnet_forward(orn.canonical_params(w, SMALL), x),
                        torch_resnet(w, x, SMALL))]
        for k in (1, 3):
            ref = torch_resnet(loop_masked_cnn_weights(w, SMALL, table, k), x, SMALL)
            errs.append(rel_err(orn.elastic_forward(w, SMALL, table, k, x), ref))
        return max(errs)

    assert worst() < 1e-10
    monkeypatch.setattr(orn, name, mutant)
    assert worst() > 1e-6, name
