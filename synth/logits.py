"""Seeded synthetic logits for the Jensen--Shannon distance (no arithmetic of
the distance itself).

The paper measures the distance on a held-out batch of its Llama models'
outputs; those models and data are not available, so logits of the same
shape stand in: for every token position u the averaged model's logits are
N(0, scale^2) over the vocabulary plus a Zipf-like head (a few dozen tokens
lifted by head_boost / sqrt(rank)), so that a few tokens carry most of the
probability as in a language model; worker m's logits are the averaged ones
plus N(0, noise^2) (replicas that drifted apart).
"""

from __future__ import annotations

import numpy as np


def numpy_logits(M, U, K, ldk=None, dtype="f32", seed=0, scale=2.0, head=48, head_boost=8.0, noise=0.2):
    """Returns (avg [U][ldk], workers [M][U][ldk]) as float32 arrays, or uint16
    bf16 bit patterns (round to nearest even) for dtype "bf16".  Elements in
    [K, ldk) are 0."""
    import torch

    ldk = K if ldk is None else ldk
    rng = np.random.default_rng(seed)
    za = (rng.standard_normal((U, K)) * scale).astype(np.float32)
    h = min(head, K)
    lift = (head_boost / np.sqrt(1.0 + np.arange(h))).astype(np.float32)
    for u in range(U):
        za[u, rng.choice(K, h, replace=False)] += lift
    zw = (za[None] + rng.standard_normal((M, U, K)).astype(np.float32) * np.float32(noise)).astype(np.float32)
    A = np.zeros((U, ldk), np.float32)
    W = np.zeros((M, U, ldk), np.float32)
    A[:, :K], W[:, :, :K] = za, zw
    if dtype == "bf16":
        A = torch.from_numpy(A).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        W = torch.from_numpy(W).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    return A, W


def torch_logits(M, U, K, ldk=None, dtype="bf16", seed=0, scale=2.0, head=48, head_boost=8.0, noise=0.2,
                 device="cuda", chunk=64):
    """The same recipe drawn on the device with torch generators (large
    sizes), `chunk` tokens at a time: the lifted head of each token is a
    uniformly random set of `head` tokens (the first ones of a random
    permutation, taken as an argsort of uniform draws)."""
    import torch

    ldk = K if ldk is None else ldk
    pdt = torch.float32 if dtype == "f32" else torch.bfloat16
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    A = torch.zeros((U, ldk), dtype=pdt, device=device)
    W = torch.zeros((M, U, ldk), dtype=pdt, device=device)
    h = min(head, K)
    lift = head_boost / torch.sqrt(1.0 + torch.arange(h, device=device, dtype=torch.float32))
    for u0 in range(0, U, chunk):
        n = min(chunk, U - u0)
        za = torch.randn((n, K), generator=g, device=device) * scale
        idx = torch.rand((n, K), generator=g, device=device).argsort(dim=1)[:, :h]
        za.scatter_add_(1, idx, lift.expand(n, h).contiguous())
        A[u0:u0 + n, :K] = za.to(pdt)
        for m in range(M):
            W[m, u0:u0 + n, :K] = (za + torch.randn((n, K), generator=g, device=device) * noise).to(pdt)
    return A, W
