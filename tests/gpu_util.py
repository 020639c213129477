"""Helpers shared by the GPU parity tests (imported by tests only)."""
from __future__ import annotations

import sys

import numpy as np

from paper_2608_10362_amd import binding, synth


def log(msg: str):
    print(f"[gpu-test] {msg}", flush=True)
    sys.stdout.flush()


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    return torch


def u32_tensor(words: np.ndarray):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(words, dtype=np.uint32).view(np.int32)).cuda()


def f32(x):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def i32(x):
    torch = torch_cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).cuda()


def kv_to_device(arr, dtype: str):
    """A synth K/V block (float32 or bf16 bits) as a device tensor of the storage type."""
    torch = torch_cuda()
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def install_context(kv: binding.KVCache, ctx, lengths, n_layers: int, dtype: str):
    """Write a synthetic resident context (synth.make_kv_context) into a device cache."""
    for l in range(n_layers):
        for b, L in enumerate(lengths):
            if L == 0:
                continue
            kv.write_context(l, b, 0, kv_to_device(ctx[l][b]["k"], dtype), kv_to_device(ctx[l][b]["v"], dtype))


def oracle_caches(shape, n_layers: int, ctx, lengths, capacity: int):
    from oracle.model import KVCache
    caches = []
    for b, L in enumerate(lengths):
        c = KVCache(shape, n_layers, capacity)
        for l in range(n_layers):
            if L:
                c.load(l, ctx[l][b]["k"], ctx[l][b]["v"])
        c.length = int(L)
        caches.append(c)
    return caches
