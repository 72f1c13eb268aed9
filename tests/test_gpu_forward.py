"""End-to-end parity of the HIP forward (through the C ABI) with the fp64
oracle, for every DN mode of every model config, plus the prefix-read
(NaN-poison) test, mode switching and batch edge cases."""
import os

import numpy as np
import pytest

import oracle
from paper_2609_10018_amd import ffi, inputs
from paper_2609_10018_amd.inputs import CONFIGS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from gpu_util import check_top1, images_on_device, rel_err  # noqa: E402

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FP32_TOL = 1e-4
BF16_TOL = 2e-2


def golden(name):
    return np.load(os.path.join(GOLDEN, f"logits_{name}.npz"))["logits"]


class Model:
    def __init__(self, name, max_batch=None, weights=None):
        self.cfg = CONFIGS[name]
        self.w = weights if weights is not None else inputs.make_weights(self.cfg)
        self.table = inputs.make_dn_table(self.cfg)
        self.max_batch = max_batch or self.cfg.batch
        self.vit = ffi.ElasticViT(self.cfg, self.w, self.table, self.max_batch)
        self.x = inputs.make_images(self.cfg, self.max_batch)
        self.xd = images_on_device(self.cfg, self.x)

    def run(self, k, batch=None):
        batch = batch or self.max_batch
        self.vit.set_mode(k)
        logits = torch.empty((batch, self.cfg.num_classes), dtype=torch.float32, device="cuda")
        self.vit.forward(self.xd[:batch], logits)
        torch.cuda.synchronize()
        return logits.cpu().numpy()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ffi.load_library()


_models = {}


def model(name):
    if name not in _models:
        _models[name] = Model(name)
    return _models[name]


def test_tiny_fp32_all_modes():
    m = model("tiny")
    for k in range(m.table.num_modes):
        got = m.run(k)
        ref = oracle.elastic_forward(m.w, m.cfg, m.table, k, m.x)
        err = rel_err(got, ref)
        print(f"tiny mode {k}: rel err {err:.3e}")
        assert err <= FP32_TOL


@pytest.mark.parametrize("name", ["vit_ti", "vit_s", "vit_b"])
def test_bf16_all_modes_match_oracle(name):
    m = model(name)
    gold = golden(name)
    assert gold.shape == (m.table.num_modes, m.cfg.batch, m.cfg.num_classes)
    for k in range(m.table.num_modes):
        got = m.run(k)
        assert np.isfinite(got).all()
        err = rel_err(got, gold[k])
        print(f"{name} mode {k}: rel err {err:.3e}")
        assert err <= BF16_TOL
        check_top1(f"{name} mode {k}", got, gold[k])


def test_tiny_emb_fp32_all_modes():
    """Modes that also narrow the embedding (64, 48, 24 channels), fp32."""
    m = model("tiny_emb")
    for k in range(m.table.num_modes):
        got = m.run(k)
        ref = oracle.elastic_forward(m.w, m.cfg, m.table, k, m.x)
        err = rel_err(got, ref)
        print(f"tiny_emb mode {k} (d_k {m.table.n_embed[k]}): rel err {err:.3e}")
        assert err <= FP32_TOL


@pytest.mark.parametrize("name", ["vit_ti_emb", "vit_b_emb"])
def test_bf16_embed_modes_match_oracle(name):
    m = model(name)
    gold = golden(name)
    n = gold.shape[1]
    assert gold.shape == (m.table.num_modes, n, m.cfg.num_classes)
    for k in range(m.table.num_modes):
        got = m.run(k)[:n]
        assert np.isfinite(got).all()
        err = rel_err(got, gold[k])
        print(f"{name} mode {k} (d_k {m.table.n_embed[k]}): rel err {err:.3e}")
        assert err <= BF16_TOL
        check_top1(f"{name} mode {k}", got, gold[k])


def test_forward_is_deterministic_and_switch_copies_nothing():
    m = model("vit_s")
    a = m.run(2)
    wb0, sb0 = m.vit.memory_info()
    free0 = torch.cuda.mem_get_info()[0]
    for i in range(1000):
        m.vit.set_mode(i % m.table.num_modes)
    assert torch.cuda.mem_get_info()[0] == free0
    assert m.vit.memory_info() == (wb0, sb0)
    b = m.run(2)
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("batch", [1, 3, 255])
def test_vit_b_partial_batches(batch):
    m = model("vit_b")
    gold = golden("vit_b")
    for k in (0, 4):
        got = m.run(k, batch)
        assert rel_err(got, gold[k][:batch]) <= BF16_TOL


@pytest.mark.parametrize("name,batches", [("vit_ti", (1, 2, 5)), ("vit_s", (1, 3, 8)),
                                          ("vit_b", (1, 2, 8)), ("vit_b_emb", (1, 8))])
def test_small_batches(name, batches):
    """Batch 1-8 (few tiles per GEMM, so the GEMMs split K over more
    workgroups; ragged K on ViT-S and in narrow modes): every mode matches the
    oracle, and repeated calls are identical."""
    m = model(name)
    gold = golden(name)
    for batch in batches:
        for k in range(m.table.num_modes):
            got = m.run(k, batch)
            assert rel_err(got, gold[k][:batch]) <= BF16_TOL, (batch, k)
            for _ in range(3):
                np.testing.assert_array_equal(m.run(k, batch), got)


def test_forward_captured_in_hip_graphs():
    """The forward allocates, synchronises and memsets nothing, so one graph
    per mode can be captured; every replay, with eager forwards in between,
    equals the eager result."""
    m = model("vit_ti")
    batch = 8
    s = torch.cuda.Stream()
    logits = torch.empty((batch, m.cfg.num_classes), dtype=torch.float32, device="cuda")
    xd = m.xd[:batch].contiguous()
    eager = {}
    with torch.cuda.stream(s):
        for k in range(m.table.num_modes):
            m.vit.set_mode(k)
            m.vit.forward(xd, logits, s)
            s.synchronize()
            eager[k] = logits.clone()
    graphs = {}
    for k in range(m.table.num_modes):
        g = torch.cuda.CUDAGraph()
        m.vit.set_mode(k)
        with torch.cuda.graph(g, stream=s):
            m.vit.forward(xd, logits, s)
        graphs[k] = g
    torch.cuda.synchronize()
    seq = inputs.mode_sequence(40, m.table.num_modes)
    other = torch.empty_like(logits)
    for i, k in enumerate(seq):
        graphs[int(k)].replay()
        torch.cuda.synchronize()
        assert torch.equal(logits, eager[int(k)]), (i, int(k))
        with torch.cuda.stream(s):            # eager work between replays
            m.vit.set_mode(int((k + 1) % m.table.num_modes))
            m.vit.forward(xd, other, s)
        s.synchronize()


def test_full_batch_forwards_repeat_and_capture():
    """ViT-B at its full batch of 256: the handle chose at create, per mode,
    tile plans and whether to run as two halves on two streams.  Every mode's
    forward repeats bit for bit, and a captured HIP graph of it (the fork to
    the handle's side stream and the join captured with it) replays the
    eager result."""
    m = model("vit_b")
    s = torch.cuda.Stream()
    logits = torch.empty((m.max_batch, m.cfg.num_classes), dtype=torch.float32, device="cuda")
    for k in range(m.table.num_modes):
        a = m.run(k)
        np.testing.assert_array_equal(m.run(k), a)
        m.vit.set_mode(k)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            m.vit.forward(m.xd, logits, s)
        for _ in range(2):
            logits.zero_()
            g.replay()
            torch.cuda.synchronize()
            np.testing.assert_array_equal(logits.cpu().numpy(), a)
        del g


def _poison_outside(w, cfg, table, k):
    """Copy of w with every weight outside mode k's active heads / units = NaN."""
    p = {key: np.array(v, copy=True) for key, v in w.items()}
    d, hd = cfg.dim, cfg.head_dim
    for l in range(cfg.depth):
        act_h, act_m = oracle.active_sets(table, k, l)
        off_h = np.setdiff1d(np.arange(cfg.heads), act_h)
        off_m = np.setdiff1d(np.arange(cfg.mlp_hidden), act_m)
        for i in off_h:
            for t in range(3):
                p["qkv_w"][l][t * d + i * hd:t * d + (i + 1) * hd] = np.nan
                p["qkv_b"][l][t * d + i * hd:t * d + (i + 1) * hd] = np.nan
            p["proj_w"][l][:, i * hd:(i + 1) * hd] = np.nan
        p["fc1_w"][l][off_m] = np.nan
        p["fc1_b"][l][off_m] = np.nan
        p["fc2_w"][l][:, off_m] = np.nan
    # embedding channels the mode drops: every tensor with a d axis
    off_e = np.setdiff1d(np.arange(d), oracle.active_embed(table, k, d))
    if off_e.size:
        p["patch_w"][off_e] = np.nan
        for key in ("patch_b", "cls", "norm_g", "norm_b"):
            p[key][off_e] = np.nan
        p["pos"][:, off_e] = np.nan
        p["head_w"][:, off_e] = np.nan
        for key in ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "proj_b", "fc2_b"):
            p[key][:, off_e] = np.nan
        p["qkv_w"][:, :, off_e] = np.nan
        p["fc1_w"][:, :, off_e] = np.nan
        p["proj_w"][:, off_e, :] = np.nan
        p["fc2_w"][:, off_e, :] = np.nan
    return p


@pytest.mark.parametrize("name,k", [("tiny", 1), ("vit_s", 3), ("vit_s", 4), ("vit_b", 4),
                                    ("tiny_emb", 2), ("vit_ti_emb", 2), ("vit_ti_emb", 3)])
def test_prefix_read_nan_poison(name, k):
    """Mode k never reads a weight outside its prefix (heads, units and
    embedding channels), ragged tails included."""
    clean = model(name)
    ref = clean.run(k)
    poisoned = Model(name, weights=_poison_outside(clean.w, clean.cfg, clean.table, k))
    got = poisoned.run(k)
    poisoned.vit.close()
    assert np.isfinite(got).all()
    np.testing.assert_array_equal(got, ref)


@pytest.mark.parametrize("name,k,batch", [("vit_s", 4, 1), ("vit_b", 4, 1), ("vit_b", 3, 8),
                                          ("vit_ti_emb", 3, 1)])
def test_prefix_read_nan_poison_small_batch(name, k, batch):
    """The split-K path of small batches (each K chunk a slice of the prefix,
    the last one ragged) reads no weight outside mode k's prefix either.  The
    reference is a clean handle of the same max_batch: handles of the same
    shapes take the same create-time plan choices (split-K ones included), so
    the two must agree bit for bit."""
    full = model(name)
    clean = Model(name, max_batch=batch, weights=full.w)
    clean.xd = full.xd[:batch].contiguous()  # the same images
    ref = clean.run(k, batch)
    clean.vit.close()
    poisoned = Model(name, max_batch=batch,
                     weights=_poison_outside(full.w, full.cfg, full.table, k))
    poisoned.xd = full.xd[:batch].contiguous()
    got = poisoned.run(k, batch)
    poisoned.vit.close()
    assert np.isfinite(got).all()
    np.testing.assert_allclose(got, ref, rtol=0, atol=0)
    # and both are the forward of the full-batch handle within bf16 rounding
    assert rel_err(got, full.run(k, batch)) <= BF16_TOL


def test_error_paths_on_device():
    m = model("tiny")
    logits = torch.empty((m.max_batch + 1, m.cfg.num_classes), device="cuda")
    big = torch.zeros((m.max_batch + 1,) + tuple(m.xd.shape[1:]), device="cuda")
    with pytest.raises(ffi.ElastoError) as e:
        m.vit.forward(big, logits)
    assert e.value.status == 7
    with pytest.raises(ffi.ElastoError) as e:
        m.vit.set_mode(m.table.num_modes)
    assert e.value.status == 6
    assert m.vit.get_mode() in range(m.table.num_modes)


@pytest.mark.parametrize("name", ["vit_b", "vit_b_emb", "tiny_emb"])
def test_mode_info_matches_cost_model(name):
    from paper_2609_10018_amd import cost
    m = model(name)
    for k in range(m.table.num_modes):
        f, wbytes = m.vit.mode_info(k)
        assert f == pytest.approx(cost.flops_per_image(m.cfg, m.table, k), rel=1e-12)
        eb = 2 if m.cfg.dtype == inputs.BF16 else 4
        assert wbytes == eb * cost.active_weight_elems(m.cfg, m.table, k)
