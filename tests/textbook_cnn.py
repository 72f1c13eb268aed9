"""A textbook bottleneck-ResNet forward from torch CPU fp64 library ops (test
helper, independent of the oracle): F.conv2d, F.relu, F.max_pool2d,
adaptive average pooling and F.linear.  Used only to pin the oracle."""
import numpy as np
import torch
import torch.nn.functional as F


def t64(a):
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def torch_resnet(w, images, cfg):
    with torch.no_grad():
        x = F.relu(F.conv2d(t64(images), t64(w["stem_w"]), t64(w["stem_b"]), stride=2, padding=3))
        x = F.max_pool2d(x, 3, stride=2, padding=1)
        for i, spec in enumerate(cfg.block_specs()):
            s = spec["stride"]
            y = F.relu(F.conv2d(x, t64(w[f"b{i}_c1_w"]), t64(w[f"b{i}_c1_b"])))
            y = F.relu(F.conv2d(y, t64(w[f"b{i}_c2_w"]), t64(w[f"b{i}_c2_b"]), stride=s,
                                padding=1))
            y = F.conv2d(y, t64(w[f"b{i}_c3_w"]), t64(w[f"b{i}_c3_b"]))
            if f"b{i}_dn_w" in w:
                x = F.conv2d(x, t64(w[f"b{i}_dn_w"]), t64(w[f"b{i}_dn_b"]), stride=s)
            x = F.relu(y + x)
        feat = F.adaptive_avg_pool2d(x, 1).flatten(1)
        return F.linear(feat, t64(w["fc_w"]), t64(w["fc_b"])).numpy()


def loop_masked_cnn_weights(w, cfg, table, k):
    """Zero every pruned filter of mode k, kernel by kernel (brute-force form
    of Eq. 7): its own kernels and bias, and the kernels that read it."""
    out = {key: np.array(v, dtype=np.float64, copy=True) for key, v in w.items()}
    for i, spec in enumerate(cfg.block_specs()):
        n = int(table.n_width[k][i])
        keep1 = set(int(c) for c in table.order1[i][:n])
        keep2 = set(int(c) for c in table.order2[i][:n])
        for c in range(spec["width"]):
            if c not in keep1:
                out[f"b{i}_c1_w"][c] = 0.0
                out[f"b{i}_c1_b"][c] = 0.0
                out[f"b{i}_c2_w"][:, c] = 0.0
            if c not in keep2:
                out[f"b{i}_c2_w"][c] = 0.0
                out[f"b{i}_c2_b"][c] = 0.0
                out[f"b{i}_c3_w"][:, c] = 0.0
    return out
