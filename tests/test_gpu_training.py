"""A training chunk with the library's own forward and backward: adapters fitted
by plain SGD to the outputs of target adapters (the frozen base shared), on
mixed-adapter batches. The loss 0.5 * ||y - y*||^2 must fall steadily: the
gradients are the right ones to train with, not only equal to the oracle's."""
import math

import numpy as np
import pytest
import torch

import paper_2608_15241_amd as lk
from tests.gpu_helpers import say

pytestmark = pytest.mark.gpu


def _bf16(t):
    return t.to(torch.bfloat16).contiguous()


@pytest.mark.parametrize("T", [200, 600])
def test_sgd_with_the_library_gradients_fits_the_target_adapters(T):
    say("training chunk", T)
    g = torch.Generator(device="cuda").manual_seed(T)
    K, N, n_ad, r = 256, 256, 3, 8
    W = _bf16(torch.randn(N, K, device="cuda", generator=g) * 0.02)
    # scales that keep the curvature along A and along B of order one
    A_true = torch.randn(n_ad, r, K, device="cuda", generator=g) / math.sqrt(K)
    B_true = torch.randn(n_ad, N, r, device="cuda", generator=g) / math.sqrt(N)
    # float32 master weights of the trained adapters (A near the target, B at
    # zero as LoRA starts), bf16 copies for the kernels
    A = A_true + 0.5 * torch.randn(n_ad, r, K, device="cuda", generator=g) / math.sqrt(K)
    B = torch.zeros(n_ad, N, r, device="cuda")
    ranks = torch.full((n_ad,), r, dtype=torch.int32, device="cuda")
    lr = 1.0
    losses = []
    for step in range(30):
        x = _bf16(torch.randn(T, K, device="cuda", generator=g))
        idx = torch.randint(0, n_ad, (T,), device="cuda", generator=g, dtype=torch.int32)
        scale = torch.ones(T, device="cuda")
        y_star = lk.local_lora_linear(x, W, _bf16(A_true), _bf16(B_true), ranks, idx, scale)
        y = lk.local_lora_linear(x, W, _bf16(A), _bf16(B), ranks, idx, scale)
        diff = y.float() - y_star.float()
        losses.append(0.5 * float((diff * diff).sum()) / T)
        dA, dB = lk.local_lora_grad(x, _bf16(diff), _bf16(A), _bf16(B), ranks, idx, scale)
        A -= lr * dA / T
        B -= lr * dB / T
    torch.cuda.synchronize()
    say("loss", ["%.4g" % v for v in losses[::5]], "->", "%.4g" % losses[-1])
    assert all(np.isfinite(losses))
    assert losses[-1] < 0.2 * losses[0], losses
    # steadily: every block of five steps ends lower than it started
    assert all(losses[i + 5] < losses[i] for i in range(0, 25, 5)), losses
