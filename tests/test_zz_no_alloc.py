"""mlp_train_step_static (the iteration on the library's own scratch array, for callers that
cannot allocate) against mlp_train_step with a caller-owned workspace.

Both run the same kernels on the same inputs, so the parameters, bf16 copies, biases and
loss must agree bit for bit. Two calls in a row on the static scratch: the full
9216-4096-4096-1000 stack at B = 256, then a smaller network, which finds the first call's
contents in the scratch. A network whose workspace exceeds the scratch is refused before
anything is enqueued."""
import numpy as np
import pytest

from synthdata import get_config, make_mlp_inputs, scaled_mlp
from tests._util import input_on_device, make_layers

pytestmark = pytest.mark.gpu


def _state(imbd, cfg, dev, seed):
    import torch
    d = make_mlp_inputs(cfg, seed=seed)
    layers = make_layers(imbd, d, dev, cfg.dtype)
    x, _ = input_on_device(d, dev, cfg.dtype)
    lab = torch.from_numpy(d["labels"]).to(dev)
    return layers, x, lab


def _run_pair(imbd, dev, cfg, seed):
    import torch
    print(f"static scratch: {cfg.name} {cfg.dims} B={cfg.batch}", flush=True)
    net = imbd.MLP(cfg.dims, cfg.batch, cfg.dtype)
    # reference: the caller-owned workspace, filled with NaN bytes (nothing may depend on it)
    layers_a, x, lab = _state(imbd, cfg, dev, seed)
    ws = torch.full((imbd.mlp_workspace_bytes(net),), 0xFF, dtype=torch.uint8, device=dev)
    loss_a = torch.zeros(1, device=dev)
    imbd.mlp_train_step(net, layers_a, x, lab, ws, cfg.lr, loss_a)
    layers_b, _, _ = _state(imbd, cfg, dev, seed)
    loss_b = torch.full((1,), float("nan"), device=dev)
    imbd.mlp_train_step_static(net, layers_b, x, lab, cfg.lr, loss_b)
    torch.cuda.synchronize()
    assert torch.equal(loss_a, loss_b) and np.isfinite(loss_b.item())
    for la, lb in zip(layers_a, layers_b):
        for k in ("w", "w_lp", "b"):
            assert torch.equal(la[k], lb[k]), k


def test_static_scratch_matches_workspace_two_calls(imbd, dev):
    big = get_config("alexnet_fc_b256")
    assert imbd.mlp_workspace_bytes(imbd.MLP(big.dims, big.batch, "bf16")) <= imbd.IMBD_STATIC_SCRATCH_BYTES
    _run_pair(imbd, dev, big, seed=0)
    _run_pair(imbd, dev, scaled_mlp((576, 320, 256, 100), 64, "bf16"), seed=1)


def test_static_scratch_refuses_a_network_that_does_not_fit(imbd, dev):
    import torch
    cfg = scaled_mlp((9216, 4096, 4096, 1000), 2048, "bf16")
    net = imbd.MLP(cfg.dims, cfg.batch, "bf16")
    assert imbd.mlp_workspace_bytes(net) > imbd.IMBD_STATIC_SCRATCH_BYTES
    # host-side refusal: the pointers are never read, nothing is enqueued
    layers = [{"w": torch.empty(1, device=dev), "w_lp": torch.empty(1, device=dev),
               "b": torch.empty(1, device=dev)}] * 3
    with pytest.raises(imbd.ImbdError) as e:
        imbd.mlp_train_step_static(net, layers, torch.empty(1, device=dev), torch.empty(1, device=dev),
                                   0.01, torch.empty(1, device=dev))
    assert e.value.status == imbd.IMBD_EWORKSPACE
    torch.cuda.synchronize()
