"""Oracle encoder (Sec. 3.2.1; architecture Sec. 4.5, App. A) pinned against
PyTorch's own Linear / BatchNorm1d(eval) / ReLU modules in fp64 and against
closed forms."""
import numpy as np
import pytest
import torch

import oracle as O


def _torch_mlp(weights, biases, bn=None):
    layers = []
    for l, (w, b) in enumerate(zip(weights, biases)):
        lin = torch.nn.Linear(w.shape[1], w.shape[0]).double()
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(w.astype(np.float64)))
            lin.bias.copy_(torch.from_numpy(b.astype(np.float64)))
        layers.append(lin)
        if l + 1 < len(weights):
            if bn is not None:
                m = torch.nn.BatchNorm1d(w.shape[0]).double().eval()
                g, beta, mu, var = bn[l]
                with torch.no_grad():
                    m.weight.copy_(torch.from_numpy(g)); m.bias.copy_(torch.from_numpy(beta))
                    m.running_mean.copy_(torch.from_numpy(mu)); m.running_var.copy_(torch.from_numpy(var))
                layers.append(m)
            layers.append(torch.nn.ReLU())
    return torch.nn.Sequential(*layers)


@pytest.mark.parametrize("widths", [(32, 64, 8), (128, 96, 64, 22), (16, 4)])
def test_encoder_matches_torch_modules_fp32_input(oracle_lib, widths):
    rng = np.random.default_rng(0)
    ws = [(rng.standard_normal((widths[i + 1], widths[i])) / np.sqrt(widths[i])).astype(np.float32)
          for i in range(len(widths) - 1)]
    bs = [rng.standard_normal(widths[i + 1]).astype(np.float32) * 0.1 for i in range(len(widths) - 1)]
    x = rng.standard_normal((37, widths[0])).astype(np.float32)
    got = O.encode(O.Encoder(ws, bs), x)
    ref = _torch_mlp(ws, bs)(torch.from_numpy(x.astype(np.float64))).detach().numpy()
    # fp64 accumulation rounded once to fp32: within one fp32 ulp of PyTorch's
    # fp64 result (the two fp64 sums may differ in their last bits)
    assert np.all(np.abs(got.astype(np.float64) - ref) <= np.spacing(np.abs(got)).astype(np.float64))


def test_encoder_batchnorm_eval_folding(oracle_lib):
    rng = np.random.default_rng(1)
    widths = (24, 40, 12)
    ws = [rng.standard_normal((widths[i + 1], widths[i])).astype(np.float32) * 0.2 for i in range(2)]
    bs = [rng.standard_normal(widths[i + 1]).astype(np.float32) * 0.1 for i in range(2)]
    g = rng.uniform(0.5, 1.5, 40); beta = rng.standard_normal(40) * 0.1
    mu = rng.standard_normal(40) * 0.2; var = rng.uniform(0.5, 2.0, 40)
    eps = 1e-5
    scale = (g / np.sqrt(var + eps)).astype(np.float32)
    shift = (beta - mu * g / np.sqrt(var + eps)).astype(np.float32)
    x = rng.standard_normal((20, 24)).astype(np.float32)
    got = O.encode(O.Encoder(ws, bs, [scale], [shift]), x)
    ref = _torch_mlp(ws, bs, bn=[(g, beta, mu, var)])(torch.from_numpy(x.astype(np.float64))).detach().numpy()
    # scale/shift are rounded to fp32, so compare at fp32 precision
    assert np.allclose(got, ref, rtol=1e-5, atol=1e-5)


def test_encoder_uint8_scaling_identity_layers(oracle_lib):
    # W = I, zero bias: logits = relu(x / 255) passed through the identity
    d = 16
    eye = np.eye(d, dtype=np.float32)
    x = np.arange(d * 3, dtype=np.uint8).reshape(3, d) * 5
    got = O.encode(O.Encoder([eye, eye], [np.zeros(d, np.float32)] * 2, input_scale=1.0 / 255.0), x)
    assert np.array_equal(got, (x.astype(np.float64) / 255.0).astype(np.float32))
    # a negative weight is cut by the ReLU of the hidden layer
    got2 = O.encode(O.Encoder([-eye, eye], [np.zeros(d, np.float32)] * 2, input_scale=1.0 / 255.0), x)
    assert np.array_equal(got2, np.zeros_like(got2))


def test_encoder_magnitude_bounds_logit(oracle_lib):
    rng = np.random.default_rng(2)
    ws = [rng.standard_normal((8, 6)).astype(np.float32), rng.standard_normal((3, 8)).astype(np.float32)]
    bs = [np.zeros(8, np.float32), rng.standard_normal(3).astype(np.float32)]
    x = rng.standard_normal((5, 6)).astype(np.float32)
    lg, mag = O.encode(O.Encoder(ws, bs), x, with_mag=True)
    assert np.all(np.abs(lg) <= mag * (1 + 1e-6))
    h = np.maximum(x.astype(np.float64) @ ws[0].T.astype(np.float64), 0)
    assert np.allclose(mag, np.abs(h[:, None, :] * ws[1][None].astype(np.float64)).sum(-1) + np.abs(bs[1]))
