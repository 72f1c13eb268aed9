"""The run-time selection loop on the GPU: elasto_profile_modes measures every
mode, its table feeds elasto_select_mode (Eq. 11), and the choice agrees with
the oracle's selection on the same measured table."""
import math

import numpy as np
import pytest

import oracle
from paper_2609_10018_amd import ffi, inputs
from paper_2609_10018_amd.inputs import CONFIGS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from gpu_util import images_on_device  # noqa: E402


@pytest.fixture(scope="module")
def vit_ti():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = CONFIGS["vit_ti"]
    w = inputs.make_weights(cfg)
    table = inputs.make_dn_table(cfg)
    vit = ffi.ElasticViT(cfg, w, table, cfg.batch)
    xd = images_on_device(cfg, inputs.make_images(cfg, cfg.batch))
    logits = torch.empty((cfg.batch, cfg.num_classes), dtype=torch.float32, device="cuda")
    yield cfg, table, vit, xd, logits
    vit.close()


def expected_memory(cfg, table, k, batch):
    """Resident bytes of mode k at this batch, as the header defines them."""
    d, T, hd, L = cfg.dim, cfg.tokens, cfg.head_dim, cfg.depth
    h, m = table.n_heads[k], table.n_mlp[k]
    mat = d * cfg.patch_k + cfg.num_classes * d + sum(4 * hd * h[l] * d + 2 * d * m[l]
                                                      for l in range(L))
    vec = 2 * d + T * d + 2 * d + cfg.num_classes + sum(
        2 * d + 3 * hd * h[l] + d + 2 * d + m[l] + d for l in range(L))
    rows = batch * T
    act = (2 * rows * d + rows * 3 * hd * max(h) + rows * hd * max(h) + rows * max(m)
           + batch * d) * 2 + batch * d * 4
    return mat * 2 + vec * 4 + act


def test_profile_modes_table(vit_ti):
    cfg, table, vit, xd, logits = vit_ti
    vit.set_mode(2)
    lat, mem, fl = vit.profile_modes(xd, logits, warmup=2, iters=7)
    assert vit.get_mode() == 2                                   # mode left as it was
    assert np.all(lat > 0) and np.all(np.isfinite(lat))
    for k in range(table.num_modes):
        assert fl[k] == pytest.approx(vit.mode_info(k)[0] * cfg.batch, rel=1e-12)
        assert mem[k] == expected_memory(cfg, table, k, cfg.batch)
    assert np.all(np.diff(mem) <= 0)                             # nested DNs: never larger
    assert lat[0] > lat[-1]                                      # 2.5 vs 0.76 GFLOP per image
    # the measured table drives Eq. 11 exactly as the oracle reads it
    for L_d in [lat.min() * 0.5, lat[1], lat[0] * 2, math.inf]:
        for A_min in [-math.inf, 0.7, 0.9]:
            acc = np.array([0.92, 0.9, 0.8, 0.7])
            want = oracle.select_dn(fl, lat, mem, acc, None, L_d=L_d, A_min=A_min)
            got = ffi.select_mode(fl, lat, mem, acc, max_latency_ms=L_d, min_accuracy=A_min)
            assert got == want


def test_profile_modes_rejects_bad_batch(vit_ti):
    cfg, table, vit, xd, logits = vit_ti
    big = torch.empty((cfg.batch + 1,) + tuple(xd.shape[1:]), dtype=xd.dtype, device="cuda")
    with pytest.raises(ffi.ElastoError) as e:
        vit.profile_modes(big, logits)
    assert e.value.status == 7
